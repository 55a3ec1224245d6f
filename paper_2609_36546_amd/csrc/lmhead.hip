// LM head + vocabulary log-softmax + top-K support for gfx950, without
// writing the logits to memory.
//
// The verifier's next-token distribution at each window row (temperature 1)
// gives the proposed token's log-prob, the LSE, the argmax, the top-K support
// of the coverage rule (Eq. (5)) and the entropy.
//
// Kernel 1 (GEMM + epilogue).  logits^T = W . hidden^T with
// v_mfma_f32_32x32x16_bf16 (fp32: 32x32x2; A = 32 vocabulary rows of W, B =
// 32 hidden rows).  A workgroup owns 256 vocabulary entries x a tile of
// hidden rows, and wave (wv, wr) owns 128 of the entries (one record group)
// x a slice of the rows.  For bf16, lmhead_gemm_dlds_kernel streams both
// operands straight into a 4-deep LDS ring of 32-channel stages, with eight
// waves (two per SIMD; four for 64- and 192-row tiles), and keeps its
// workgroups resident, each walking tiles; lmhead_gemm_kernel (fp32) stages
// 32 channels through registers, double buffered, with four waves.  In the
// accumulator layout a lane holds one hidden row and 16 vocabulary entries
// per 32x32 block, so every per-row reduction over the vocabulary is in-lane
// plus one exchange with lane l^32.  For each (row, 128-entry group) the
// epilogue emits a record: the three largest logits with their indices, the
// fourth largest value, sum exp(l - v1) over each 32-entry quarter and over
// the group, and sum exp(l - v1) * l.
//
// Kernel 2 (merge, one workgroup per row).  LSE = M + log sum_g s_g e^(v1_g-M),
// entropy = LSE - (sum_g e_g e^(v1_g-M)) / (sum_g s_g e^(v1_g-M)).  Top-K: the
// K best of the recorded top-3 candidates; a group with three picks whose
// recorded fourth value reaches the K-th pick may hide further members, so
// such a group's logits are recomputed exactly and the selection is redone --
// the result is the exact top-K of all V logits (ties: lower index first).
// The proposal's logit is one dot product.
//
// Kernel 3 (draws, sample_kernel): a categorical draw from a row's
// distribution by inverse CDF over the group records, then the selected
// group's quarter sums, then 32 recomputed logits -- the takeover replacement
// of Eq. (9) and the proposer's per-row draw.  logp_gather_kernel gives the
// log-probs of a row at listed indices (the other model's top-K support).
#include "common.h"
#include "kernels.h"

namespace ipdv {
namespace {

constexpr int kVT = 256;      // vocabulary entries per workgroup
constexpr int kGroup = 128;   // vocabulary entries per record (one wave's share)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct LmParams {
  const void* hidden;
  const void* hidden_tiled;   // bf16 hidden rows in W's tiled block layout (workspace copy)
  const void* W;
  const int32_t* prop_tok;
  const int32_t* out_rows;
  int M, Hd, V, K;
  int w_tiled;        // W in 16-row x 32-channel blocks (lmhead_pack_w), else [V][Hd]
  int n_groups, n_rt, n_vt;
  int rec_stride;          // record entries per row: n_groups rounded up to a multiple of 4
  int vt_base, n_vt_run;   // this launch's vocabulary tiles: vt_base .. vt_base + n_vt_run - 1
  // Group records, [M][rec_stride] each: the three largest logits of the group,
  // their positions in it (rec_i: 7 bits each, i1 | i2 << 7 | i3 << 14; any
  // value where the logit is -inf), the fourth largest value, sum exp(l - v1) over each
  // 32-entry quarter of the group (rec_sq[q]: entries 32 q .. 32 q + 31), over
  // the group (rec_s, the quarters added in pairs) and sum exp(l - v1) * l
  // over the group.
  float* rec_v1;
  float* rec_v2;
  float* rec_v3;
  float* rec_v4;
  float* rec_sq[4];
  float* rec_s;
  float* rec_e;
  int32_t* rec_i;
  float* lse;
  float* logp_prop;
  int32_t* argmax;
  int32_t* topk_idx;
  float* topk_logp;
  float* entropy;
};

// Element offset of W[v][c]: row-major [V][Hd], or tiled in 1 KB blocks of
// 16 rows x 32 channels, [ceil(V/16)][Hd/32][16][32] (lmhead_pack_w).  A
// 16-byte chunk (8 channels from a multiple of 8) is contiguous either way.
__device__ __forceinline__ size_t w_off(const LmParams& p, int v, int c) {
  return p.w_tiled ? ((size_t)(v >> 4) * (p.Hd >> 5) + (c >> 5)) * 512 + (v & 15) * 32 + (c & 31)
                   : (size_t)v * p.Hd + c;
}

// W [V][Hd] -> [ceil(V/16)][Hd/32][16][32]: one thread per 16-byte chunk of
// the output, in output order (rows past V are zero).
__global__ __launch_bounds__(256) void pack_w_kernel(const bf16* W, int V, int Hd, bf16* Wt,
                                                     size_t n_chunks) {
  // n_chunks < 2^31 (the host checks), so the index math is 32-bit
  const unsigned t = blockIdx.x * 256u + threadIdx.x;
  if (t >= n_chunks) return;
  const unsigned blk = t >> 6;               // 64 chunks per 1 KB block
  const int within = (int)(t & 63);
  const unsigned nb_c = (unsigned)Hd >> 5;
  const int v = (int)(blk / nb_c) * 16 + (within >> 2);
  const int c = (int)(blk % nb_c) * 32 + (within & 3) * 8;
  typedef __attribute__((__vector_size__(16))) int i32x4;
  i32x4 x = {0, 0, 0, 0};
  if (v < V) x = ld16<i32x4>(W + (size_t)v * Hd + c);
  *reinterpret_cast<i32x4*>(Wt + (size_t)t * 8) = x;
}

// MFMA flavour of the register-staged kernel (fp32; bf16 always takes the
// direct-to-LDS kernel).  STAGE = hidden channels per pipeline stage;
// a lane supplies its k-step operand from channels koff(ks, h) of the stage
// (h = lane / 32).  Any bijection works as long as A and B agree.
template <typename DT> struct Mm;

template <> struct Mm<float> {
  static constexpr int STAGE = 32;
  static constexpr int KSTEPS = STAGE / 2;
  typedef float frag;
  __device__ static floatx16 mma(frag a, frag b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static int koff(int ks, int h) { return 16 * h + ks; }
};

// (value desc, index asc) order: true if (a, ia) ranks before (b, ib).
__device__ __forceinline__ bool before(float a, int ia, float b, int ib) {
  // bitwise, not short-circuit: compares and selects, no branches in loops
  return (a > b) | ((a == b) & (ia < ib));
}

// Top-3 (value desc, index asc) insertion of (x, ix), with the fourth value:
// (v1, i1) >= (v2, i2) >= (v3, i3) >= v4.
__device__ __forceinline__ void top3_push(float x, int ix, float& v1, int& i1, float& v2, int& i2,
                                          float& v3, int& i3, float& v4) {
  const bool c1 = before(x, ix, v1, i1);
  const bool c2 = before(x, ix, v2, i2);
  const bool c3 = before(x, ix, v3, i3);
  v4 = __builtin_amdgcn_fmed3f(v3, v4, x);
  const float nv3 = c2 ? v2 : (c3 ? x : v3);
  const int ni3 = c2 ? i2 : (c3 ? ix : i3);
  const float nv2 = c1 ? v1 : (c2 ? x : v2);
  const int ni2 = c1 ? i1 : (c2 ? ix : i2);
  v1 = c1 ? x : v1;
  i1 = c1 ? ix : i1;
  v2 = nv2;
  i2 = ni2;
  v3 = nv3;
  i3 = ni3;
}

typedef __attribute__((__vector_size__(16))) int i32x4;

// Offset of register e of 32x32 block vb from the lane's first vocabulary
// entry: block vb covers 32 entries, register e entry 8 (e / 4) + e % 4 (plus
// 4 for the upper half-wave).  Local index j = 16 vb + e.
__device__ __forceinline__ constexpr int epi_off(int j) {
  return 32 * (j >> 4) + 8 * ((j >> 2) & 3) + (j & 3);
}

// Epilogue: per hidden row (lane column) and this wave's 128 vocabulary
// entries, the group record (top-3 with indices, fourth value, s, e).  A lane
// holds 64 of the group's entries for its row, in increasing vocabulary order
// along j, so a later equal value never displaces an earlier one and the
// running top-4 needs no index comparisons: three medians of three and a
// select keep the values, three compares and five selects the local indices.
// The partner lane (l ^ 32) holds the other 64.  FULL: every entry of the tile
// is < V (no masking).
template <int RB, bool FULL>
__device__ __forceinline__ void lm_epilogue(const LmParams& p, floatx16 (&acc)[4][RB], int vt, int m0,
                                            int wv, int wr) {
  const int lane = lane_id();
  const int h = lane >> 5;
  const int vlane = vt * kVT + kGroup * wv + 4 * h;   // entry of local index 0
  const int g = vt * (kVT / kGroup) + wv;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int m = m0 + 32 * RB * wr + 32 * rb + (lane & 31);
    if (!FULL) {
#pragma unroll
      for (int j = 0; j < 64; ++j)
        acc[j >> 4][rb][j & 15] = (vlane + epi_off(j) < p.V) ? acc[j >> 4][rb][j & 15] : -INFINITY;
    }
    float v1 = -INFINITY, v2 = -INFINITY, v3 = -INFINITY, v4 = -INFINITY;
    int j1 = 0, j2 = 0, j3 = 0;
    bool ranked = false;
    if (FULL) {
      // Values first: each entry is clamped into the sorted top-4.
#pragma unroll
      for (int j = 0; j < 64; ++j) {
        const float x = acc[j >> 4][rb][j & 15];
        v4 = __builtin_amdgcn_fmed3f(v3, v4, x);
        v3 = __builtin_amdgcn_fmed3f(v2, v3, x);
        v2 = __builtin_amdgcn_fmed3f(v1, v2, x);
        // a plain v_max: fmaxf (or a med3 against infinity) would add a
        // NaN-quieting max per entry
        asm("v_max_f32 %0, %1, %2" : "=v"(v1) : "v"(v1), "v"(x));
        // v4 here, entry by entry: left to itself the compiler keeps every
        // intermediate v3 in a register of its own and builds v4 later
        asm volatile("" : "+v"(v4));
      }
      // Equal values among a lane's top three anywhere in the wave send the
      // wave through the single-pass ranking below.
      ranked = __builtin_amdgcn_ballot_w64((v1 == v2) | (v2 == v3)) == 0;
    }
    if (ranked) {
      // Then the indices.  With v1 > v2 > v3 the first two values occur once
      // and v3 may recur (an equal later entry ranks behind the first), so
      // the first entry holding each value is its index: a downward scan
      // keeps the lowest.
#pragma unroll
      for (int j = 63; j >= 0; --j) {
        const float x = acc[j >> 4][rb][j & 15];
        j1 = (x == v1) ? j : j1;
        j2 = (x == v2) ? j : j2;
        j3 = (x == v3) ? j : j3;
        // one entry at a time: hoisted compares would each hold a lane mask
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      v1 = v2 = v3 = v4 = -INFINITY;
      j1 = j2 = j3 = 0;
#pragma unroll
      for (int j = 0; j < 64; ++j) {
        const float x = acc[j >> 4][rb][j & 15];
        const bool c1 = x > v1, c2 = x > v2, c3 = x > v3;
        v4 = __builtin_amdgcn_fmed3f(v3, v4, x);
        v3 = __builtin_amdgcn_fmed3f(v2, v3, x);
        v2 = __builtin_amdgcn_fmed3f(v1, v2, x);
        v1 = c1 ? x : v1;   // a select on c1: fmaxf would add a NaN-quieting max per entry
        j3 = c2 ? j2 : (c3 ? j : j3);
        j2 = c1 ? j1 : (c2 ? j : j2);
        j1 = c1 ? j : j1;
      }
    }
    int i1 = (v1 == -INFINITY) ? 0x7fffffff : vlane + epi_off(j1);
    int i2 = (v2 == -INFINITY) ? 0x7fffffff : vlane + epi_off(j2);
    int i3 = (v3 == -INFINITY) ? 0x7fffffff : vlane + epi_off(j3);
    {
      // merge the partner lane's top-3: the fourth of the union is the max of
      // the fourth after pushing its top-3 and its own fourth
      const float ov1 = lane_xor32(v1), ov2 = lane_xor32(v2);
      const float ov3 = lane_xor32(v3), ov4 = lane_xor32(v4);
      const int oi1 = lane_xor32(i1), oi2 = lane_xor32(i2);
      const int oi3 = lane_xor32(i3);
      top3_push(ov1, oi1, v1, i1, v2, i2, v3, i3, v4);
      top3_push(ov2, oi2, v1, i1, v2, i2, v3, i3, v4);
      top3_push(ov3, oi3, v1, i1, v2, i2, v3, i3, v4);
      v4 = fmaxf(v4, ov4);
    }
    // v1 is now the group maximum; exp-sum and entropy numerator against it
    const float mub = ((v1 == -INFINITY) ? 0.f : v1) * kLog2e;
    // block vb of the accumulators is the group's quarter vb (32 entries)
    float sq[4] = {0.f, 0.f, 0.f, 0.f}, ee = 0.f;
#pragma unroll
    for (int j = 0; j < 64; ++j) {
      const float x = acc[j >> 4][rb][j & 15];
      const float pe = fast_exp2(fmaf(x, kLog2e, -mub));
      sq[j >> 4] += pe;
      if (FULL)
        ee = fmaf(pe, x, ee);
      else
        ee += (x != -INFINITY) ? pe * x : 0.f;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) sq[q] += lane_xor32(sq[q]);
    ee += lane_xor32(ee);
    if (h == 0 && m < p.M && g < p.n_groups) {
      const size_t r = (size_t)m * p.rec_stride + g;
      p.rec_v1[r] = v1;
      p.rec_v2[r] = v2;
      p.rec_v3[r] = v3;
      p.rec_v4[r] = v4;
#pragma unroll
      for (int q = 0; q < 4; ++q) p.rec_sq[q][r] = (v1 == -INFINITY) ? 0.f : sq[q];
      p.rec_s[r] = (v1 == -INFINITY) ? 0.f : (sq[0] + sq[1]) + (sq[2] + sq[3]);
      p.rec_e[r] = (v1 == -INFINITY) ? 0.f : ee;
      const int gb = kGroup * g;   // the group's first entry
      p.rec_i[r] = ((i1 - gb) & 127) | (((i2 - gb) & 127) << 7) | (((i3 - gb) & 127) << 14);
    }
  }
}

template <int RB>
__device__ __forceinline__ void lm_epilogue_any(const LmParams& p, floatx16 (&acc)[4][RB], int vt,
                                                int m0, int wv, int wr) {
  if ((vt + 1) * kVT <= p.V)
    lm_epilogue<RB, true>(p, acc, vt, m0, wv, wr);
  else
    lm_epilogue<RB, false>(p, acc, vt, m0, wv, wr);
}

// Tile number id.  The hardware deals workgroup ids to the 8 XCDs
// round-robin (id % 8), and a persistent workgroup steps its tile number by
// the grid size, a multiple of 8, so it stays on its XCD.  XCD x takes a
// contiguous range of vocabulary tiles, and the row tiles of one vocabulary
// tile run side by side on it: the W tile they share is fetched from HBM
// once into that XCD's L2, and every 64-byte line of the group records (16
// groups = 8 vocabulary tiles of one row) is completed inside one L2 before
// it is written back.  A launch covers the vocabulary tiles vt_base ..
// vt_base + n_vt_run - 1, as tile numbers below ceil(n_vt_run / 8) * 8 * n_rt;
// the others are empty (false).
__device__ __forceinline__ bool gemm_tile(const LmParams& p, int id, int& vt, int& rt) {
  const int xcd = id & 7, local = id >> 3;
  const int per = p.n_vt_run / 8, extra = p.n_vt_run % 8;
  const int j = local / p.n_rt;
  if (j >= per + (xcd < extra ? 1 : 0)) return false;
  vt = p.vt_base + xcd * per + min(xcd, extra) + j;
  rt = local % p.n_rt;
  return true;
}

template <typename DT, int RB>
__global__ __launch_bounds__(256) void lmhead_gemm_kernel(LmParams p) {
  int vt, rt;
  if (!gemm_tile(p, blockIdx.x, vt, rt)) return;
  typedef Mm<DT> MM;
  constexpr int NM = 64 * RB;                       // hidden rows per workgroup
  constexpr int LDW = MM::STAGE + 16 / (int)sizeof(DT);   // LDS row pitch (elements)
  constexpr int EPL = 16 / (int)sizeof(DT);         // elements per 16-byte load
  constexpr int CPR = MM::STAGE / EPL;              // 16-byte chunks per row and stage
  constexpr int NLW = kVT * CPR / 256;              // W loads per thread and stage
  constexpr int NLH = NM * CPR / 256;               // hidden loads per thread and stage
  const int m0 = rt * NM;
  const int v0 = vt * kVT;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int wv = w & 1, wr = w >> 1;
  const int lane = lane_id();
  const int h = lane >> 5;

  __shared__ __attribute__((aligned(16))) DT s_w[2][kVT * LDW];
  __shared__ __attribute__((aligned(16))) DT s_h[2][NM * LDW];

  const DT* Wp = reinterpret_cast<const DT*>(p.W);
  const DT* Hp = reinterpret_cast<const DT*>(p.hidden);
  i32x4 rw[NLW], rh[NLH];
  const int nst = p.Hd / MM::STAGE;

  auto load_stage = [&](int k0) {
#pragma unroll
    for (int u = 0; u < NLW; ++u) {
      const int e = tid + 256 * u;
      const int r = e / CPR, c = e % CPR;
      const int v = min(v0 + r, p.V - 1);           // rows past V: any valid row, masked later
      rw[u] = ld16<i32x4>(Wp + (size_t)v * p.Hd + k0 + EPL * c);
    }
#pragma unroll
    for (int u = 0; u < NLH; ++u) {
      const int e = tid + 256 * u;
      const int r = e / CPR, c = e % CPR;
      const int m = min(m0 + r, p.M - 1);           // rows past M: any valid row, never read
      rh[u] = ld16<i32x4>(Hp + (size_t)m * p.Hd + k0 + EPL * c);
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int u = 0; u < NLW; ++u) {
      const int e = tid + 256 * u;
      *reinterpret_cast<i32x4*>(&s_w[buf][(e / CPR) * LDW + EPL * (e % CPR)]) = rw[u];
    }
#pragma unroll
    for (int u = 0; u < NLH; ++u) {
      const int e = tid + 256 * u;
      *reinterpret_cast<i32x4*>(&s_h[buf][(e / CPR) * LDW + EPL * (e % CPR)]) = rh[u];
    }
  };

  floatx16 acc[4][RB];
#pragma unroll
  for (int vb = 0; vb < 4; ++vb)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[vb][rb][e] = 0.f;

  load_stage(0);
  store_stage(0);
  for (int st = 0; st < nst; ++st) {
    const bool more = st + 1 < nst;
    if (more) load_stage((st + 1) * MM::STAGE);
    __syncthreads();
    const DT* sw = s_w[st & 1] + (128 * wv + (lane & 31)) * LDW;
    const DT* sh = s_h[st & 1] + (32 * RB * wr + (lane & 31)) * LDW;
#pragma unroll
    for (int ks = 0; ks < MM::KSTEPS; ++ks) {
      const int ko = MM::koff(ks, h);
      typename MM::frag a[4], b[RB];
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) a[vb] = *reinterpret_cast<const typename MM::frag*>(sw + 32 * vb * LDW + ko);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) b[rb] = *reinterpret_cast<const typename MM::frag*>(sh + 32 * rb * LDW + ko);
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = MM::mma(a[vb], b[rb], acc[vb][rb]);
    }
    if (more) store_stage((st + 1) & 1);
  }

  lm_epilogue_any<RB>(p, acc, vt, m0, wv, wr);
}

// ---------------------------------------------------------------------------
// bf16 GEMM with direct-to-LDS operand loads (global_load_lds_dwordx4).
//
// Each 16-byte load lands straight in LDS (lane i of an instruction fills
// bytes 16 i .. 16 i + 15 of a 1 KB block), so no registers stage the tiles.
// In a 4-deep LDS ring of 32-channel stages, two stages are in flight while
// one is multiplied and the one before it is still being read.  Rows are 64 bytes; the 16-byte chunk c of row r sits
// at position c ^ ((r / 4) % 4), which puts the 16 rows an MFMA operand read
// touches in distinct bank groups; the loading lane fetches the global chunk
// that belongs at its position.
// ---------------------------------------------------------------------------

constexpr int kDStage = 32;   // hidden channels per stage (64 bytes per row)

__device__ __forceinline__ int dl_off(int r, int c) { return 64 * r + 16 * (c ^ ((r >> 2) & 3)); }

template <int RB, int NBUF, int NW>
__global__ __launch_bounds__(64 * NW) void lmhead_gemm_dlds_kernel(LmParams p) {
  static_assert(NBUF >= 3 && NBUF <= 5, "ring depth");
  static_assert(NW == 4 || NW == 8, "2 x (NW / 2) waves");
  int id = blockIdx.x, vt, rt;
  if (!gemm_tile(p, id, vt, rt)) return;
  constexpr int NM = 32 * RB * (NW / 2);        // hidden rows per workgroup
  constexpr int WB = kVT * 64;                  // W tile bytes per stage
  constexpr int SB = WB + NM * 64;              // stage bytes
  constexpr int NBLK = (kVT + NM) / 16;         // 1 KB load blocks per stage
  constexpr int PW = NBLK / NW;                 // load instructions per wave and stage
  constexpr int KS = kDStage / 16;              // MFMA k-steps per stage
  static_assert(KS == 2 && (NBUF - 2) * PW <= 63 && NBLK % NW == 0, "pipeline shape");
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int wv = w & 1, wr = w >> 1;
  const int lane = lane_id();
  const int h = lane >> 5;
  const int rr = lane & 31;
  const int nst = p.Hd / kDStage;

  __shared__ __attribute__((aligned(1024))) char s_ring[NBUF * SB];

  const bf16* Wp = reinterpret_cast<const bf16*>(p.W);
  const bf16* Hp = reinterpret_cast<const bf16*>(p.hidden_tiled);
  // This lane's source row and chunk for each of its load blocks, for tile
  // (vt_, rt_).
  const bf16* src[PW];
  auto set_src = [&](int vt_, int rt_) {
    const int m0 = rt_ * NM, v0 = vt_ * kVT;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int u = w + NW * j;
      const int r = (u < kVT / 16 ? 16 * u : 16 * (u - kVT / 16)) + (lane >> 2);
      const int c = (lane & 3) ^ ((r >> 2) & 3);
      if (u < kVT / 16) {
        if (p.w_tiled) {
          // the stage's 16 rows x 32 channels are one 1 KB block; the lane takes
          // the same row and (swizzled) chunk as in the row-major case, so the
          // LDS image is identical.  Blocks past V: any valid block, masked later.
          const int vb = min((v0 >> 4) + u, ((p.V + 15) >> 4) - 1);
          src[j] = Wp + (size_t)vb * (p.Hd >> 5) * 512 + (lane >> 2) * 32 + 8 * c;
        } else {
          const int v = min(v0 + r, p.V - 1);     // rows past V: any valid row, masked later
          src[j] = Wp + (size_t)v * p.Hd + 8 * c;
        }
      } else {
        // hidden rows come from the per-call copy in the same 16-row x 32-channel
        // block layout (rows past M there are zero and never stored)
        const int mb = min((m0 >> 4) + (u - kVT / 16), ((p.M + 15) >> 4) - 1);
        src[j] = Hp + (size_t)mb * (p.Hd >> 5) * 512 + (lane >> 2) * 32 + 8 * c;
      }
    }
  };
  set_src(vt, rt);
  // Stage st goes to buffer st % NBUF.  Stages past the end reload the last
  // one into a free buffer, so that every wave has the same number of loads
  // in flight at every boundary.  dma(st, j0, j1): this wave's load blocks
  // [j0, j1) of stage st.
  // Load blocks j < kVT / (16 NW) are W (for every wave); a stage advances a tiled
  // block (W when packed, the hidden copy always) by 512 elements per 32 channels.
  const int wk = p.w_tiled ? 16 : 1;
  auto dma = [&](int st, int j0, int j1) {
    char* buf = s_ring + (st % NBUF) * SB;
    const int k0 = min(st, nst - 1) * kDStage;
#pragma unroll
    for (int j = j0; j < j1; ++j)
      dma16(src[j] + (j < kVT / (16 * NW) ? wk : 16) * k0, buf + 1024 * (w + NW * j));
  };
  // Operand offsets of this lane within a stage.  Chunk 2 ks + h of a row sits
  // at 16 ((2 ks + h) ^ q), q = row bits 2-3, which is the ks = 0 offset xor
  // 32 ks; 32-row steps keep q.
  const int a_off = dl_off(128 * wv + rr, h);
  const int b_off = WB + dl_off(32 * RB * wr + rr, h);
  bf16x8 fa[2][4], fb[2][RB];
  auto load = [&](int set, const char* buf, int ks) {
    const int x = 32 * ks;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
      fb[set][rb] = *reinterpret_cast<const bf16x8*>(buf + ((b_off + 2048 * rb) ^ x));
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
      fa[set][vb] = *reinterpret_cast<const bf16x8*>(buf + ((a_off + 2048 * vb) ^ x));
  };

  floatx16 acc[4][RB];
  // MFMAs of operand set `set` over vocabulary block vb.
  auto mma = [&](int set, int vb) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
      acc[vb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[set][vb], fb[set][rb], acc[vb][rb], 0, 0, 0);
  };
#define IPDV_SB __builtin_amdgcn_sched_barrier(0)

  // Boundary into stage b, between the two k-steps of stage b - 1: each wave
  // waits for its own loads of b (NBUF - 3 later stages may stay in flight),
  // the barrier makes every wave's visible, and buffer (b - 2) % NBUF starts
  // refilling with stage b + NBUF - 2.  Every wave has consumed stage b - 2:
  // it waited for that stage's last operands before its second k-step's
  // MFMAs, which precede this barrier.  Stage b - 1 may still be read (its
  // second k-step's operands can be in flight), so it is not refilled yet.  A
  // bare s_barrier: the fence of __syncthreads would wait for every stage in
  // flight.  The operand reads of a k-step are issued one k-step of MFMAs
  // ahead of their use (stage b's first k-step right after the boundary, its
  // second at the top of stage b), the hidden fragments first, since every
  // MFMA of the k-step needs them.  The refill's loads are spread over the
  // MFMAs (a burst of them stalls the issuing wave, and that idles its share
  // of the matrix pipe).  sched_barrier pins the order.
  //
  // The workgroup is persistent: after a tile's last MFMAs it waits for the
  // reloads past the end, and once every wave is done with the ring it
  // issues the first NBUF - 1 stages of its next tile, whose loads land while
  // the finished tile's epilogue runs.  The next tile's first wait is then a
  // full one: the epilogue's record stores are in flight too, and loads and
  // stores are not promised to complete in issue order.
  constexpr int Q1 = PW / 4, Q2 = PW / 2, Q3 = 3 * PW / 4;   // refill split points
#pragma unroll
  for (int s0 = 0; s0 < NBUF - 1; ++s0) dma(s0, 0, PW);
  bool first = true;
  for (;;) {
    if (first)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NBUF - 2) * PW) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    load(0, s_ring, 0);
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[vb][rb][e] = 0.f;
    for (int st = 0; st + 1 < nst; ++st) {
      const char* cur = s_ring + (st % NBUF) * SB;
      const int pend = st + NBUF - 2;            // refill started at the last boundary
      load(1, cur, 1);
      IPDV_SB;
      mma(0, 0);
      IPDV_SB;
      if (st > 0) dma(pend, Q1, Q2);
      IPDV_SB;
      mma(0, 1);
      IPDV_SB;
      if (st > 0) dma(pend, Q2, Q3);
      IPDV_SB;
      mma(0, 2);
      IPDV_SB;
      if (st > 0) dma(pend, Q3, PW);
      IPDV_SB;
      mma(0, 3);
      IPDV_SB;
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NBUF - 3) * PW) : "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      dma(pend + 1, 0, Q1);
      load(0, s_ring + ((st + 1) % NBUF) * SB, 0);
      IPDV_SB;
      mma(1, 0);
      mma(1, 1);
      mma(1, 2);
      mma(1, 3);
      IPDV_SB;
    }
    {
      const char* cur = s_ring + ((nst - 1) % NBUF) * SB;
      load(1, cur, 1);
      mma(0, 0);
      mma(0, 1);
      mma(0, 2);
      mma(0, 3);
      mma(1, 0);
      mma(1, 1);
      mma(1, 2);
      mma(1, 3);
    }
    // the reloads past the end, and this wave's last operand reads
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");

    const int vt_done = vt, m0_done = rt * NM;
    id += gridDim.x;
    const bool more = gemm_tile(p, id, vt, rt);
    if (more) {
      __builtin_amdgcn_s_barrier();   // every wave is done with the ring
      asm volatile("" ::: "memory");
      set_src(vt, rt);
#pragma unroll
      for (int s0 = 0; s0 < NBUF - 1; ++s0) dma(s0, 0, PW);
    }
    lm_epilogue_any<RB>(p, acc, vt_done, m0_done, wv, wr);
    if (!more) break;
    // the load addresses again, rather than held in registers across the epilogue
    set_src(vt, rt);
    first = false;
  }
#undef IPDV_SB
}

// ---------------------------------------------------------------------------
// Merge: one workgroup (256 threads) per row.
// ---------------------------------------------------------------------------

constexpr int kMT = 256;

// Block sums of three values at once (s holds 3 * waves floats).
__device__ void block_sum3(float& a, float& b, float& c, float* s) {
  a = wave_sum(a);
  b = wave_sum(b);
  c = wave_sum(c);
  constexpr int NW = kMT / kWave;
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if (lane_id() == 0) { s[w] = a; s[NW + w] = b; s[2 * NW + w] = c; }
  __syncthreads();
  a = b = c = 0.f;
  for (int ww = 0; ww < NW; ++ww) { a += s[ww]; b += s[NW + ww]; c += s[2 * NW + ww]; }
}

__device__ float block_max(float x, float* s) {
  x = wave_max(x);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if (lane_id() == 0) s[w] = x;
  __syncthreads();
  float t = -INFINITY;
  for (int ww = 0; ww < kMT / kWave; ++ww) t = fmaxf(t, s[ww]);
  return t;
}

// Candidates per row: three per group plus every element of the groups whose
// third-best made it into the list.  Such a group contributes three entries
// to a K-entry list, so at most K/3 groups are ever recomputed.
constexpr int kMaxSplit = IPDV_MAX_K_DEV / 3;
constexpr int kSplitCand = kMaxSplit * kGroup;

// Groups per merge thread held in registers: V <= kMT * kMaxGPT * kGroup.
constexpr int kMaxGPT = 8;
constexpr int kCPG = 3;        // candidates per group (its recorded top-3)

// One reduction step: combine with the (value, index) DPP moves in from
// another lane; lanes without a source keep theirs.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ void best_step(float& v, int& ix) {
  const float ov = __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(-INFINITY), __float_as_int(v),
                                                              CTRL, ROW_MASK, 0xf, false));
  const int oi = __builtin_amdgcn_update_dpp(0x7fffffff, ix, CTRL, ROW_MASK, 0xf, false);
  if (before(ov, oi, v, ix)) { v = ov; ix = oi; }
}

// Wave-wide best (value desc, index asc) of one candidate per lane, returned
// to every lane: DPP row shifts 1/2/4/8 and row broadcasts 15/31 carry the
// best towards lane 63 (a few cycles per step, no LDS round trip).
__device__ __forceinline__ void wave_best(float& v, int& ix) {
  best_step<0x111, 0xf>(v, ix);   // row_shr:1
  best_step<0x112, 0xf>(v, ix);   // row_shr:2
  best_step<0x114, 0xf>(v, ix);   // row_shr:4
  best_step<0x118, 0xf>(v, ix);   // row_shr:8
  best_step<0x142, 0xa>(v, ix);   // row_bcast:15 into rows 1, 3
  best_step<0x143, 0xc>(v, ix);   // row_bcast:31 into rows 2, 3
  v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
  ix = __builtin_amdgcn_readlane(ix, 63);
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

// Top-K of the n <= kMT entries of an LDS list with distinct indices, by
// rank: thread t takes entry t and counts the entries before it in the
// (value desc, index asc) order, reading the list as LDS broadcasts; an entry
// of rank r < K goes to position r.  Positions without an entry get
// (-inf, 0x7fffffff).  NaN values are never picked and precede nothing.
// All threads of the block take part (two barriers).
__device__ __forceinline__ void block_topk_rank(const float* lv, const int* li, int n, int K,
                                                float* out_v, int* out_i) {
  const int tid = threadIdx.x;
  if (tid < K) {
    out_v[tid] = -INFINITY;
    out_i[tid] = 0x7fffffff;
  }
  __syncthreads();
  if (tid < n) {
    const float v = lv[tid];
    const int i = li[tid];
    if (v == v) {
      // 16-byte broadcast reads of four entries at a time; entries past n
      // (any contents) are excluded by their position
      int r = 0;
#pragma unroll 4
      for (int c = 0; c < n; c += 4) {
        const floatx4 y = *reinterpret_cast<const floatx4*>(lv + c);
        const i32x4 yi = *reinterpret_cast<const i32x4*>(li + c);
#pragma unroll
        for (int e = 0; e < 4; ++e) r += ((c + e < n) & before(y[e], yi[e], v, i)) ? 1 : 0;
      }
      if (r < K) {
        out_v[r] = v;
        out_i[r] = i;
      }
    }
  }
  __syncthreads();
}

constexpr int kCap = 2048;     // survivor list capacity (candidates >= theta)
constexpr int kMaxHd = 4096;   // hidden sizes the merge can stage in LDS for recomputes

template <typename DT> struct Frag16;
template <> struct Frag16<bf16> { typedef bf16x8 type; };
template <> struct Frag16<float> { typedef floatx4 type; };

// Exact logits of n vocabulary entries, vocab_of(e) for e < n (entries past V
// give -inf), for the hidden row staged in s_hid (fp32).  A wave takes NB entries at a time and lane l covers channels
// EPL l + 64 EPL i of each, so one load instruction reads 64 consecutive
// 16-byte chunks of a W row and the loads of all NB entries (4 chunks each)
// are in flight together; a shuffle reduction finishes each dot product.
template <typename DT, int NB, typename VOCAB>   // NB: entries per wave and batch
__device__ void recompute_entries(const LmParams& p, const float* s_hid, int n, VOCAB vocab_of,
                                  float* out_v, int* out_i) {
  typedef typename Frag16<DT>::type frag;
  const DT* Wp = reinterpret_cast<const DT*>(p.W);
  constexpr int EPL = 16 / (int)sizeof(DT);
  constexpr int NP = 4;                       // chunks per lane and entry in flight
  constexpr int NW = kMT / kWave;
  const int lane = lane_id(), wv = threadIdx.x / kWave;
  for (int e0 = wv * NB; e0 < n; e0 += NW * NB) {
    float acc[NB];
    int vv[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      vv[b] = vocab_of(min(e0 + b, n - 1));
      acc[b] = 0.f;
    }
    for (int c0 = 0; c0 < p.Hd; c0 += NP * kWave * EPL) {
      frag w[NB][NP];
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < NP; ++i) {
          // out-of-range rows and channels load a valid chunk; it is masked below
          const int c = min(c0 + EPL * (lane + kWave * i), p.Hd - EPL);
          w[b][i] = ld16<frag>(Wp + w_off(p, min(vv[b], p.V - 1), c));
        }
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        const int c = c0 + EPL * (lane + kWave * i);
        if (c < p.Hd) {
          float hv[EPL];
#pragma unroll
          for (int e = 0; e < EPL; ++e) hv[e] = s_hid[c + e];
#pragma unroll
          for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[b] = fmaf(to_f32(w[b][i][e]), hv[e], acc[b]);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      float a = acc[b];
      a = wave_sum(a);
      if (lane == 0 && e0 + b < n) {
        const bool ok = vv[b] < p.V;
        out_v[e0 + b] = ok ? a : -INFINITY;
        out_i[e0 + b] = ok ? vv[b] : 0x7fffffff;
      }
    }
  }
}

// The 128 logits of each listed group (split groups of the merge).
template <typename DT, int NB = 4>
__device__ void recompute_logits(const LmParams& p, const float* s_hid, const int* s_split, int ns,
                                 float* out_v, int* out_i) {
  recompute_entries<DT, NB>(p, s_hid, ns * kGroup,
                            [&](int e) { return s_split[e / kGroup] * kGroup + e % kGroup; },
                            out_v, out_i);
}

template <typename DT>
__global__ __launch_bounds__(kMT) void lmhead_merge_kernel(LmParams p) {
  const int m = blockIdx.x;
  const int tid = threadIdx.x;
  const int wv = tid >> 6;
  const int lane = lane_id();
  const int G = p.n_groups;
  const int K = p.K;
  const size_t base = (size_t)m * p.rec_stride;
  constexpr int NW = kMT / kWave;
  __shared__ float s_red[3 * NW];
  __shared__ float s_theta[NW];
  __shared__ __attribute__((aligned(16))) float s_tm[kMT];   // thread maxima (theta)
  __shared__ float s_wv[NW][IPDV_MAX_K_DEV];
  __shared__ int s_wi[NW][IPDV_MAX_K_DEV];
  __shared__ float s_top_v[IPDV_MAX_K_DEV];
  __shared__ int s_top_i[IPDV_MAX_K_DEV];
  __shared__ int s_split[kMaxSplit];
  __shared__ int s_nsplit, s_n;
  __shared__ __attribute__((aligned(16))) float s_lv[kCap];   // survivors, then survivors + recomputed logits
  __shared__ __attribute__((aligned(16))) int s_li[kCap];
  __shared__ float s_cv[kSplitCand];    // recomputed logits of split groups
  __shared__ int s_ci[kSplitCand];
  __shared__ float s_hid[kMaxHd];       // the row's hidden state, for recomputes
  __shared__ float s_lv2[kCap];         // survivor list after a recompute
  __shared__ int s_li2[kCap];

  // The proposal's logit is one dot product; its loads go out first so that
  // their latency overlaps the record loads and reductions.
  typedef typename Frag16<DT>::type frag;
  constexpr int EPL = 16 / (int)sizeof(DT);
  constexpr int NPC = kMaxHd / (EPL * kMT);   // chunks of the dot product per thread
  const int pv = p.prop_tok[m];
  const bool pok = pv >= 0 && pv < p.V;
  frag ph[NPC], pw[NPC];
  {
    const DT* hr = reinterpret_cast<const DT*>(p.hidden) + (size_t)m * p.Hd;
    const DT* wr = reinterpret_cast<const DT*>(p.W);
#pragma unroll
    for (int u = 0; u < NPC; ++u) {
      const int k = min(EPL * (tid + kMT * u), p.Hd - EPL);   // past Hd: masked below
      ph[u] = ld16<frag>(hr + k);
      pw[u] = ld16<frag>(wr + w_off(p, pok ? pv : 0, k));
    }
  }

  // This thread's groups (register resident): slot u holds group
  // merge_group(u) = 4 kMT (u / 4) + 4 tid + u % 4, so each record field of
  // four consecutive groups arrives in one 16-byte load.
  float cv[kCPG * kMaxGPT];
  int ci[kCPG * kMaxGPT];
  float rs[kMaxGPT], re[kMaxGPT];
  float mx = -INFINITY;
#pragma unroll
  for (int blk = 0; blk < kMaxGPT / 4; ++blk) {
    const int g4 = 4 * kMT * blk + 4 * tid;
    const bool ok4 = g4 < G;
    // loads are unconditional (a group past G reads group 0 of the row, or
    // the padding of the last four; both are masked below)
    const size_t o = base + (ok4 ? g4 : 0);
    const floatx4 v1 = ld16<floatx4>(p.rec_v1 + o);
    const floatx4 v2 = ld16<floatx4>(p.rec_v2 + o);
    const floatx4 v3 = ld16<floatx4>(p.rec_v3 + o);
    const i32x4 ix = ld16<i32x4>(p.rec_i + o);
    const floatx4 sg = ld16<floatx4>(p.rec_s + o);
    const floatx4 ee = ld16<floatx4>(p.rec_e + o);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int u = 4 * blk + e;
      const bool ok = g4 + e < G;
      cv[kCPG * u] = ok ? v1[e] : -INFINITY;
      cv[kCPG * u + 1] = ok ? v2[e] : -INFINITY;
      cv[kCPG * u + 2] = ok ? v3[e] : -INFINITY;
      // indices from the group's first entry and the packed positions; an
      // entry holding -inf has none
      const int gb = kGroup * (g4 + e);
      ci[kCPG * u] = (ok & (v1[e] != -INFINITY)) ? gb + (ix[e] & 127) : 0x7fffffff;
      ci[kCPG * u + 1] = (ok & (v2[e] != -INFINITY)) ? gb + ((ix[e] >> 7) & 127) : 0x7fffffff;
      ci[kCPG * u + 2] = (ok & (v3[e] != -INFINITY)) ? gb + ((ix[e] >> 14) & 127) : 0x7fffffff;
      rs[u] = ok ? sg[e] : 0.f;
      re[u] = ok ? ee[e] : 0.f;
      mx = fmaxf(mx, cv[kCPG * u]);
    }
  }
  if (tid == 0) { s_n = 0; s_nsplit = 0; }

  // Log-sum-exp and entropy sums (group maxima are the v1 records).
  const float M = block_max(mx, s_red);
  const float Mu = (M == -INFINITY) ? 0.f : M;
  float S = 0.f, E = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxGPT; ++u) {
    const int gi = 4 * kMT * (u / 4) + 4 * tid + u % 4;
    if (gi < G) {
      const float wgt = fast_exp2((cv[kCPG * u] - Mu) * kLog2e);
      S += rs[u] * wgt;
      E += re[u] * wgt;
    }
  }
  float PD = 0.f;
#pragma unroll
  for (int u = 0; u < NPC; ++u)
    if (EPL * (tid + kMT * u) < p.Hd) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) PD = fmaf(to_f32(ph[u][e]), to_f32(pw[u][e]), PD);
    }
  block_sum3(S, E, PD, s_red);
  const float lse = Mu + fast_log2(S) * kLn2;

  // theta: a lower bound of the K-th largest logit.  The K largest lane
  // maxima of a wave are K distinct logits, so the K-th largest of them bounds
  // the K-th largest logit from below; theta is the best of the waves'
  // bounds.  Each lane ranks its maximum against the wave's 64 (16-byte
  // broadcast LDS reads; ties by lane), and the lane of rank K - 1 publishes.
  if (lane == 0) s_theta[wv] = -INFINITY;
  s_tm[tid] = mx;
  __syncthreads();
  {
    const float* wm = s_tm + kWave * wv;
    int r = 0;
#pragma unroll
    for (int c = 0; c < kWave; c += 4) {
      const floatx4 y = *reinterpret_cast<const floatx4*>(wm + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) r += before(y[e], c + e, mx, lane) ? 1 : 0;
    }
    if (r == K - 1) s_theta[wv] = mx;
  }
  __syncthreads();
  float theta = s_theta[0];
  for (int w2 = 1; w2 < NW; ++w2) theta = fmaxf(theta, s_theta[w2]);
  // survivors: candidates >= theta, compacted with one LDS atomic per wave
  // (a wave prefix of the per-thread counts places each thread's run)
  {
    int cnt = 0;
#pragma unroll
    for (int c = 0; c < kCPG * kMaxGPT; ++c) cnt += ((ci[c] != 0x7fffffff) & (cv[c] >= theta)) ? 1 : 0;
    const int incl = wave_incl_scan_i(cnt);
    const int wtot = __builtin_amdgcn_readlane(incl, kWave - 1);
    int wbase = 0;
    if (lane == 0 && wtot > 0) wbase = atomicAdd(&s_n, wtot);
    int slot = __builtin_amdgcn_readlane(wbase, 0) + incl - cnt;
#pragma unroll
    for (int c = 0; c < kCPG * kMaxGPT; ++c) {
      if ((ci[c] != 0x7fffffff) & (cv[c] >= theta)) {
        if (slot < kCap) { s_lv[slot] = cv[c]; s_li[slot] = ci[c]; }
        ++slot;
      }
    }
  }
  __syncthreads();
  // Many ties at theta: select from all records instead of the list.
  bool overflow = s_n > kCap;
  int n_list = min(s_n, kCap);

  // Exact top-K.  Round 0 picks from the candidates; a group with three picks
  // may hide a fourth member, so its logits are recomputed and round 1 picks
  // again (then every element left out ranks after the K-th pick).
  for (int round = 0; round < 2; ++round) {
    const int ns = s_nsplit;
    if (overflow) {
      wave_topk(cv, ci, s_cv, s_ci, ns * kGroup, K, s_wv[wv], s_wi[wv]);
      __syncthreads();
      if (wv == 0) {
        float xv0 = -INFINITY, xv1 = -INFINITY;
        int xi0 = 0x7fffffff, xi1 = 0x7fffffff;
        if (lane < NW * K) { xv0 = s_wv[lane / K][lane % K]; xi0 = s_wi[lane / K][lane % K]; }
        if (lane + kWave < NW * K) {
          xv1 = s_wv[(lane + kWave) / K][(lane + kWave) % K];
          xi1 = s_wi[(lane + kWave) / K][(lane + kWave) % K];
        }
        const float fv[2] = {xv0, xv1};
        const int fi[2] = {xi0, xi1};
        wave_topk(fv, fi, s_cv, s_ci, 0, K, s_top_v, s_top_i);
      }
    } else if (n_list <= kMT) {
      block_topk_rank(s_lv, s_li, n_list, K, s_top_v, s_top_i);
    } else if (wv == 0) {
      const float none[1] = {-INFINITY};
      const int nonei[1] = {0x7fffffff};
      wave_topk(none, nonei, s_lv, s_li, n_list, K, s_top_v, s_top_i);
    }
    __syncthreads();
    if (round == 1) break;
    // Groups picked three times whose fourth value reaches the K-th pick may
    // hide further members: only those are recomputed.  Pick a checks its
    // group when it is the group's first pick and two later picks share it.
    if (tid < K) {
      const int ia = s_top_i[tid];
      const int ga = (int)((unsigned)ia / kGroup);
      bool first = ia != 0x7fffffff;
      int later = 0;
      for (int b2 = 0; b2 < K; ++b2) {
        const int ib = s_top_i[b2];
        const bool same = (b2 != tid) & (ib != 0x7fffffff) & ((int)((unsigned)ib / kGroup) == ga);
        first &= !(same & (b2 < tid));
        later += (same & (b2 > tid)) ? 1 : 0;
      }
      if (first && later >= kCPG - 1 && p.rec_v4[base + ga] >= s_top_v[K - 1]) {
        const int slot = atomicAdd(&s_nsplit, 1);
        if (slot < kMaxSplit) s_split[slot] = ga;
      }
    }
    __syncthreads();
    const int nsplit = min(s_nsplit, kMaxSplit);
    if (nsplit == 0) break;
    {
      const DT* hr = reinterpret_cast<const DT*>(p.hidden) + (size_t)m * p.Hd;
      for (int k = tid; k < p.Hd; k += kMT) s_hid[k] = to_f32(hr[k]);
      __syncthreads();
      recompute_logits<DT>(p, s_hid, s_split, nsplit, s_cv, s_ci);
    }
    __syncthreads();
    bool from_records = overflow;
    if (!overflow) {
      // survivors of split groups are replaced by the recomputed values; when
      // the kept survivors and the recomputed logits together exceed the
      // list, round 1 selects from all records instead
      if (tid == 0) s_n = 0;
      __syncthreads();
      for (int c = tid; c < n_list; c += kMT) {
        bool sp = false;
        for (int t = 0; t < nsplit; ++t) sp |= (s_li[c] / kGroup == s_split[t]);
        if (!sp) {
          const int slot = atomicAdd(&s_n, 1);
          if (slot < kCap) { s_lv2[slot] = s_lv[c]; s_li2[slot] = s_li[c]; }
        }
      }
      __syncthreads();
      const int kept = s_n;
      if (kept + nsplit * kGroup <= kCap) {
        for (int c = tid; c < nsplit * kGroup; c += kMT) {
          s_lv2[kept + c] = s_cv[c];
          s_li2[kept + c] = s_ci[c];
        }
        __syncthreads();
        n_list = kept + nsplit * kGroup;
        for (int c = tid; c < n_list; c += kMT) { s_lv[c] = s_lv2[c]; s_li[c] = s_li2[c]; }
      } else {
        from_records = true;
      }
    }
    if (from_records) {
      // drop the split groups' records: their members now come from s_cv
      overflow = true;
#pragma unroll
      for (int u = 0; u < kMaxGPT; ++u) {
        const int gi = 4 * kMT * (u / 4) + 4 * tid + u % 4;
        bool sp = false;
        for (int t = 0; t < nsplit; ++t) sp |= (s_split[t] == gi);
        if (sp) {
#pragma unroll
          for (int c = 0; c < kCPG; ++c) {
            cv[kCPG * u + c] = -INFINITY;
            ci[kCPG * u + c] = 0x7fffffff;
          }
        }
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
  if (tid == 0) p.logp_prop[orow] = pok ? PD - lse : NAN;
}

// ---------------------------------------------------------------------------
// Draws from softmax(l) at temperature 1 (Appendix A): the takeover
// replacement (Eq. (9), second case; one workgroup per sequence) and the
// proposer's per-row draw (one workgroup per row).  The inverse CDF over the
// vocabulary in index order is taken in three levels: the group records give
// each 128-entry group's mass, exp(v1_g - max) times its quarter sums, so a
// block-wide prefix scan over the groups finds the group the uniform falls
// in; the group's four quarter sums find the 32-entry quarter, at the same
// fraction of the group's mass; the quarter's 32 logits are recomputed
// exactly and the draw finishes inside it.
// ---------------------------------------------------------------------------

struct SampleParams {
  const int32_t* seq_ids;
  const int32_t* cu_q;
  const uint8_t* driver;
  const int32_t* event_row;
  const int32_t* row_local;
  const float* u;
  int32_t eos_id;
  int32_t* token;
  uint8_t* finished;
};

// Inclusive prefix sum over the block (thread order); *total gets the sum.
__device__ float block_scan(float x, float* s_w, float* total) {
  const int lane = lane_id(), w = threadIdx.x / kWave;
  constexpr int NW = kMT / kWave;
  x = wave_incl_scan(x);
  __syncthreads();
  if (lane == kWave - 1) s_w[w] = x;
  __syncthreads();
  float before = 0.f, all = 0.f;
  for (int ww = 0; ww < NW; ++ww) {
    before += ww < w ? s_w[ww] : 0.f;
    all += s_w[ww];
  }
  *total = all;
  return x + before;
}

// PER_ROW: one draw per hidden row m (blockIdx.x), with u[m], into token[m].
// Otherwise: one workgroup per handled sequence b; only a student-driven
// window with a takeover draws, at the takeover row, with u[b], into token[b]
// (and a drawn EOS finishes the sequence).
template <typename DT, bool PER_ROW>
__global__ __launch_bounds__(kMT) void sample_kernel(LmParams p, SampleParams s) {
  constexpr int NW = kMT / kWave;
  const int tid = threadIdx.x;
  __shared__ float s_red[3 * NW];
  __shared__ float s_hid[kMaxHd];
  __shared__ int s_g[1];
  __shared__ int s_first, s_last;
  __shared__ float s_cv[32];
  __shared__ int s_ci[32];
  __shared__ float s_gq[4];
  int b, m;
  if (PER_ROW) {
    b = m = blockIdx.x;
  } else {
    b = s.seq_ids ? s.seq_ids[blockIdx.x] : blockIdx.x;
    const int ev = s.event_row[b];
    const int r = ev >= 0 ? s.cu_q[b] + ev : -1;
    m = r < 0 ? -1 : (s.row_local ? s.row_local[r] : r);
    // only student-driven windows with an event (a takeover) draw
    if (s.driver[b] != 0 || ev < 0 || m < 0 || m >= p.M) {
      if (tid == 0) s.token[b] = -1;
      return;
    }
  }
  const int G = p.n_groups;
  const size_t base = (size_t)m * p.rec_stride;
  // Thread t holds the records of groups [t per, (t+1) per) in registers, per
  // a multiple of 4 (16-byte loads); the hidden row is staged in LDS
  // meanwhile (for the recompute below).
  const int per = ((G + kMT - 1) / kMT + 3) / 4 * 4;   // <= kMaxGPT (V <= kMT kMaxGPT kGroup)
  const int g0 = tid * per;
  float v1r[kMaxGPT], wr[kMaxGPT], qr[4][kMaxGPT];   // qr: each group's quarter sums
#pragma unroll
  for (int blk = 0; blk < kMaxGPT / 4; ++blk) {
    const int g4 = g0 + 4 * blk;
    const bool ok4 = 4 * blk < per && g4 < G;
    const size_t o = base + (ok4 ? g4 : 0);   // unconditional loads, masked below
    const floatx4 v1 = ld16<floatx4>(p.rec_v1 + o);
    const floatx4 q0 = ld16<floatx4>(p.rec_sq[0] + o);
    const floatx4 q1 = ld16<floatx4>(p.rec_sq[1] + o);
    const floatx4 q2 = ld16<floatx4>(p.rec_sq[2] + o);
    const floatx4 q3 = ld16<floatx4>(p.rec_sq[3] + o);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool ok = ok4 && g4 + e < G;
      v1r[4 * blk + e] = ok ? v1[e] : -INFINITY;
      wr[4 * blk + e] = ok ? (q0[e] + q1[e]) + (q2[e] + q3[e]) : 0.f;
      qr[0][4 * blk + e] = q0[e];
      qr[1][4 * blk + e] = q1[e];
      qr[2][4 * blk + e] = q2[e];
      qr[3][4 * blk + e] = q3[e];
    }
  }
  {
    const DT* hr = reinterpret_cast<const DT*>(p.hidden) + (size_t)m * p.Hd;
    for (int k = tid; k < p.Hd; k += kMT) s_hid[k] = to_f32(hr[k]);
  }
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < kMaxGPT; ++i) mx = fmaxf(mx, v1r[i]);
  mx = block_max(mx, s_red);
  float mine = 0.f;                              // this thread's mass
#pragma unroll
  for (int i = 0; i < kMaxGPT; ++i) {
    wr[i] = v1r[i] != -INFINITY ? wr[i] * fast_exp2((v1r[i] - mx) * kLog2e) : 0.f;
    mine += wr[i];
  }
  float tot;
  const float incl = block_scan(mine, s_red, &tot);
  const float t = s.u[b] * tot;
  // the thread whose range holds t walks its groups in order; if rounding put
  // t above every cumulative sum, the last group with mass is taken
  if (tid == 0) { s_first = kMT; s_last = -1; s_g[0] = -1; }
  __syncthreads();
  {
    // one LDS atomic per wave: its first thread whose range passes t, its
    // last thread with mass
    const unsigned long long m_in = __ballot(mine > 0.f && incl > t);
    const unsigned long long m_nz = __ballot(mine > 0.f);
    const int w0 = tid & ~(kWave - 1);
    if (lane_id() == 0 && m_in) atomicMin(&s_first, w0 + __builtin_ctzll(m_in));
    if (lane_id() == 0 && m_nz) atomicMax(&s_last, w0 + 63 - __builtin_clzll(m_nz));
  }
  __syncthreads();
  const int owner = s_first < kMT ? s_first : s_last;
  if (tid == owner) {
    // walk this thread's groups in order: the first whose cumulative mass
    // passes t; the last with mass when t is above them all (rounding)
    const bool crossing = s_first < kMT;
    float c = incl - mine;
    int gi = -1;
    float before = 0.f, w = 1.f, gq[4] = {0.f, 0.f, 0.f, 0.f};
    bool found = false;
#pragma unroll
    for (int i = 0; i < kMaxGPT; ++i) {
      if (!found && wr[i] > 0.f) {
        gi = g0 + i;
        before = c;
        w = wr[i];
#pragma unroll
        for (int q = 0; q < 4; ++q) gq[q] = qr[q][i];
        found = crossing && c + wr[i] > t;
      }
      c += wr[i];
    }
    s_g[0] = gi;
    s_red[2 * NW] = found ? fminf(fmaxf((t - before) / w, 0.f), 1.f) : 1.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) s_gq[q] = gq[q];   // the group's quarter sums, for every thread
  }
  __syncthreads();
  const int gsel = s_g[0];
  const float frac = s_red[2 * NW];
  if (gsel < 0) {                  // no mass at all (cannot happen for finite logits)
    if (tid == 0) s.token[b] = -1;
    return;
  }
  // the quarter of the group (32 entries) holding the draw, from its sums
  const float q0 = s_gq[0], q1 = s_gq[1], q2 = s_gq[2], q3 = s_gq[3];
  const float qs[4] = {q0, q1, q2, q3};
  const float tq = frac * ((q0 + q1) + (q2 + q3));
  // first quarter whose cumulative sum passes tq; the last with mass when
  // rounding leaves tq above them all
  int qsel = 0;
  float qbefore = 0.f, cq = 0.f;
  bool qfound = false;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (!qfound && qs[q] > 0.f) {
      qsel = q;
      qbefore = cq;
      qfound = cq + qs[q] > tq;
    }
    cq += qs[q];
  }
  const float frac2 = qfound ? fminf(fmaxf((tq - qbefore) / qs[qsel], 0.f), 1.f) : 1.f;
  const int v0 = gsel * kGroup + 32 * qsel;
  // exact logits of the quarter's 32 entries (one batch: 8 per wave), then
  // the draw inside it at the same fraction of its mass
  recompute_entries<DT, 8>(p, s_hid, 32, [&](int e) { return v0 + e; }, s_cv, s_ci);
  __syncthreads();
  if (tid < kWave) {
    const float a = tid < 32 ? s_cv[tid] : -INFINITY;
    float gm = a;
    gm = wave_max(gm);
    const float pr = a == -INFINITY ? 0.f : fast_exp2((a - gm) * kLog2e);
    const float c = wave_incl_scan(pr);
    const float S = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(c), kWave - 1));
    const float th = frac2 * S;
    const unsigned long long in = __ballot(pr > 0.f && c > th);
    const unsigned long long nz = __ballot(pr > 0.f);
    const int i = in ? __builtin_ctzll(in) : 63 - __builtin_clzll(nz);   // rounding guard
    if (tid == 0) {
      const int tok = s_ci[i];
      s.token[b] = tok;
      if (!PER_ROW && tok == s.eos_id) s.finished[b] = 1;
    }
  }
}


// GEMM launch per input type: bf16 takes the direct-to-LDS kernel when the
// hidden size is a multiple of four stages, fp32 the register-staged one.
dim3 gemm_grid(const LmParams& p) { return dim3((p.n_vt_run + 7) / 8 * 8 * p.n_rt); }

// Launch of the persistent direct-to-LDS GEMM: as many workgroups as the
// device holds at once (cached per device; a multiple of 8, so that each
// stays on its XCD), but no more than there are tile numbers.
template <int RB, int NBUF, int NW>
void launch_dlds(const LmParams& q, hipStream_t st) {
  static int slots[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = -1;
  int n = dev >= 0 ? slots[dev] : 0;
  if (n == 0) {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per_cu, reinterpret_cast<const void*>(&lmhead_gemm_dlds_kernel<RB, NBUF, NW>), 64 * NW, 0) !=
            hipSuccess ||
        per_cu < 1)
      per_cu = 1;
    n = max(8, device_cus() * per_cu / 8 * 8);
    if (dev >= 0) slots[dev] = n;
  }
  const dim3 grid((unsigned)min((int)gemm_grid(q).x, n));
  hipLaunchKernelGGL((lmhead_gemm_dlds_kernel<RB, NBUF, NW>), grid, dim3(64 * NW), 0, st, q);
}

template <int RB>
void launch_gemm(const LmParams& p, dim3 grid, hipStream_t st, bf16) {
  // 64 * RB hidden rows per workgroup.  256 and 128 rows take eight waves
  // (two per SIMD, each 128 vocabulary entries x 32 * RB / 2 rows), 64 and
  // 192 rows four.  The direct-to-LDS kernels read the hidden rows from a
  // copy in W's tiled block layout, written first into the workspace, so
  // that every operand load reads whole cache lines.
  // Hd is a multiple of 64 (the host checks), so of the 32-channel stage.
  const size_t n_chunks = (size_t)((p.M + 15) / 16) * 16 * p.Hd / 8;
  hipLaunchKernelGGL(pack_w_kernel, dim3((unsigned)((n_chunks + 255) / 256)), dim3(256), 0, st,
                     reinterpret_cast<const bf16*>(p.hidden), p.M, p.Hd,
                     reinterpret_cast<bf16*>(const_cast<void*>(p.hidden_tiled)), n_chunks);
  trace_mark(st);   // the hidden copy's interval ends here; the GEMM's begins
  if constexpr (RB == 4) {
    // With one row tile (M <= 256): 256-row tiles for as many whole rounds
    // of one tile per compute unit as the vocabulary fills; the vocabulary
    // tiles left over for a last, partial round run as 128-row tiles in a
    // second launch, which spreads that round's work over twice as many
    // compute units (M = 256: 594 tiles were 2.3 rounds).  With more row
    // tiles the single launch's own tail balancing does better than a second
    // launch after a kernel boundary (measured at M = 464 and 512).
    const int cus = device_cus();
    const int n_main = p.n_rt == 1 ? p.n_vt / cus * cus : p.n_vt;
    LmParams q = p;
    if (n_main > 0) {
      q.vt_base = 0;
      q.n_vt_run = n_main;
      launch_dlds<2, 4, 8>(q, st);
    }
    if (n_main < p.n_vt) {
      q.vt_base = n_main;
      q.n_vt_run = p.n_vt - n_main;
      q.n_rt = (p.M + 127) / 128;
      launch_dlds<1, 4, 8>(q, st);
    }
  } else if constexpr (RB == 2)
    launch_dlds<1, 4, 8>(p, st);
  else
    launch_dlds<RB, 4, 4>(p, st);
}

template <int RB>
void launch_gemm(const LmParams& p, dim3 grid, hipStream_t st, float) {
  trace_mark(st);   // no hidden copy for fp32: an empty interval
  hipLaunchKernelGGL((lmhead_gemm_kernel<float, RB>), grid, dim3(256), 0, st, p);
}

template <typename DT, int RB>
hipError_t launch_rb(const LmParams& p, hipStream_t st) {
  if ((size_t)((p.M + 15) / 16) * 16 * p.Hd / 8 >= (size_t(1) << 31)) return hipErrorInvalidValue;   // pack index range
  const dim3 grid = gemm_grid(p);
  trace_begin(st);
  launch_gemm<RB>(p, grid, st, DT{});
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  trace_mark(st);
  hipLaunchKernelGGL((lmhead_merge_kernel<DT>), dim3(p.M), dim3(kMT), 0, st, p);
  e = hipGetLastError();
  trace_mark(st);
  return e;
}

}  // namespace

// Compute units of the current device (cached per device; 256 if unknown).
int device_cus() {
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

LmPlan lm_plan(int M, int Hd, int V, int K, bool bf16) {
  LmPlan pl{};
  pl.n_groups = (V + kGroup - 1) / kGroup;
  pl.n_vt = (V + kVT - 1) / kVT;
  // 64*RB hidden rows per workgroup (RB <= 4); fp32 keeps RB = 1 so that its
  // double-buffered stage fits the LDS.
  const int rows = M < 256 ? M : 256;
  pl.rb = rows <= 64 ? 1 : rows <= 128 ? 2 : rows <= 192 ? 3 : 4;
  if (!bf16) pl.rb = 1;
  pl.n_rt = (M + 64 * pl.rb - 1) / (64 * pl.rb);
  pl.rec_stride = (pl.n_groups + 3) / 4 * 4;
  const size_t recs = (size_t)M * pl.rec_stride;
  pl.rec_bytes = recs * sizeof(float);
  pl.hid_off = 11 * ((pl.rec_bytes + 255) / 256 * 256);   // the 11 record arrays, then the hidden copy
  pl.workspace_bytes = pl.hid_off + (bf16 ? (size_t)((M + 15) / 16) * 16 * Hd * 2 : 0) + 256;
  (void)K;
  return pl;
}

namespace {

// Kernel parameters of an LM-head call: shapes, plan and the record arrays
// carved out of the workspace.
LmParams lm_params(const void* hidden, const void* W, int M, int Hd, int V, int K, const LmPlan& pl,
                   void* workspace) {
  LmParams p{};
  p.hidden = hidden;
  p.hidden_tiled = reinterpret_cast<char*>(workspace) + pl.hid_off;
  p.W = W;
  p.M = M;
  p.Hd = Hd;
  p.V = V;
  p.K = K;
  p.n_groups = pl.n_groups;
  p.rec_stride = pl.rec_stride;
  p.n_rt = pl.n_rt;
  p.n_vt = pl.n_vt;
  p.vt_base = 0;
  p.n_vt_run = pl.n_vt;
  const size_t stride = (pl.rec_bytes + 255) / 256 * 256;
  char* ws = reinterpret_cast<char*>(workspace);
  p.rec_v1 = reinterpret_cast<float*>(ws);
  p.rec_v2 = reinterpret_cast<float*>(ws + stride);
  p.rec_v3 = reinterpret_cast<float*>(ws + 2 * stride);
  p.rec_v4 = reinterpret_cast<float*>(ws + 3 * stride);
  for (int q = 0; q < 4; ++q) p.rec_sq[q] = reinterpret_cast<float*>(ws + (4 + q) * stride);
  p.rec_e = reinterpret_cast<float*>(ws + 8 * stride);
  p.rec_i = reinterpret_cast<int32_t*>(ws + 9 * stride);
  p.rec_s = reinterpret_cast<float*>(ws + 10 * stride);
  return p;
}

}  // namespace

hipError_t launch_lmhead(const LmLaunch& L, const LmPlan& pl, hipStream_t st) {
  if (L.M == 0) return hipSuccess;
  LmParams p = lm_params(L.hidden, L.W, L.M, L.Hd, L.V, L.K, pl, L.workspace);
  p.w_tiled = L.w_tiled ? 1 : 0;
  p.prop_tok = L.prop_tok;
  p.out_rows = L.out_rows;
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

namespace {

// log-softmax at listed vocabulary indices: one workgroup per row, the row's
// hidden vector staged in LDS, each wave streaming 4 W rows at a time with
// 16-byte loads across its lanes (the merge's exact recompute).
constexpr int kMaxGather = IPDV_MAX_GATHER_DEV;

template <typename DT>
__global__ __launch_bounds__(kMT) void logp_gather_kernel(LmParams p, const float* lse,
                                                          const int32_t* idx, int n, float* out) {
  const int m = blockIdx.x;
  __shared__ float s_hid[kMaxHd];
  __shared__ float s_v[kMaxGather];
  __shared__ int s_i[kMaxGather];
  const DT* hr = reinterpret_cast<const DT*>(p.hidden) + (size_t)m * p.Hd;
  for (int k = threadIdx.x; k < p.Hd; k += kMT) s_hid[k] = to_f32(hr[k]);
  __syncthreads();
  const int32_t* ir = idx + (size_t)m * n;
  // indices outside [0, V) read as V: recompute_entries gives them -inf
  recompute_entries<DT, 4>(p, s_hid, n, [&](int e) {
    const int v = ir[e];
    return (v < 0 || v >= p.V) ? p.V : v;
  }, s_v, s_i);
  __syncthreads();
  const float l = lse[m];
  for (int e = threadIdx.x; e < n; e += kMT) out[(size_t)m * n + e] = s_v[e] - l;
}

}  // namespace

hipError_t launch_logp_gather(const GatherLaunch& L, hipStream_t st) {
  if (L.M == 0 || L.n == 0) return hipSuccess;
  LmParams p{};
  p.hidden = L.hidden;
  p.W = L.W;
  p.M = L.M;
  p.Hd = L.Hd;
  p.V = L.V;
  p.w_tiled = L.w_tiled ? 1 : 0;
  trace_begin(st);
  if (L.dtype_bf16)
    hipLaunchKernelGGL((logp_gather_kernel<bf16>), dim3(L.M), dim3(kMT), 0, st, p, L.lse, L.idx,
                       L.n, L.logp);
  else
    hipLaunchKernelGGL((logp_gather_kernel<float>), dim3(L.M), dim3(kMT), 0, st, p, L.lse, L.idx,
                       L.n, L.logp);
  const hipError_t e = hipGetLastError();
  trace_mark(st);
  return e;
}

hipError_t launch_sample_rows(const SampleLaunch& L, const LmPlan& pl, hipStream_t st) {
  if (L.M == 0) return hipSuccess;
  LmParams p = lm_params(L.hidden, L.W, L.M, L.Hd, L.V, L.K, pl, const_cast<void*>(L.workspace));
  p.w_tiled = L.w_tiled ? 1 : 0;
  SampleParams s{};
  s.u = L.u;
  s.token = L.token;
  trace_begin(st);
  if (L.dtype_bf16)
    hipLaunchKernelGGL((sample_kernel<bf16, true>), dim3(L.M), dim3(kMT), 0, st, p, s);
  else
    hipLaunchKernelGGL((sample_kernel<float, true>), dim3(L.M), dim3(kMT), 0, st, p, s);
  const hipError_t e = hipGetLastError();
  trace_mark(st);
  return e;
}

hipError_t launch_sample_takeover(const SampleLaunch& L, const LmPlan& pl, hipStream_t st) {
  if (L.n_seq == 0) return hipSuccess;
  LmParams p = lm_params(L.hidden, L.W, L.M, L.Hd, L.V, L.K, pl, const_cast<void*>(L.workspace));
  p.w_tiled = L.w_tiled ? 1 : 0;
  const SampleParams s{L.seq_ids, L.cu_q, L.driver, L.event_row, L.row_local, L.u, L.eos_id, L.token,
                       L.finished};
  trace_begin(st);
  if (L.dtype_bf16)
    hipLaunchKernelGGL((sample_kernel<bf16, false>), dim3(L.n_seq), dim3(kMT), 0, st, p, s);
  else
    hipLaunchKernelGGL((sample_kernel<float, false>), dim3(L.n_seq), dim3(kMT), 0, st, p, s);
  const hipError_t e = hipGetLastError();
  trace_mark(st);
  return e;
}

hipError_t launch_pack_w(const void* W, int V, int Hd, void* W_tiled, hipStream_t st) {
  const size_t n_chunks = (size_t)((V + 15) / 16) * 16 * Hd / 8;
  if (n_chunks == 0) return hipSuccess;
  if (n_chunks >= (size_t(1) << 31)) return hipErrorInvalidValue;   // pack index range
  trace_begin(st);
  hipLaunchKernelGGL(pack_w_kernel, dim3((unsigned)((n_chunks + 255) / 256)), dim3(256), 0, st,
                     reinterpret_cast<const bf16*>(W), V, Hd, reinterpret_cast<bf16*>(W_tiled),
                     n_chunks);
  const hipError_t e = hipGetLastError();
  trace_mark(st);
  return e;
}

}  // namespace ipdv
