// MoE router (gate): for each token, expert logits from the bf16 hidden
// state and the bf16 router weight, sigmoid scores, group-limited top-k
// selection and normalised weights (the gating step before the token sort;
// the paper's Background on Mixture-of-Experts names top-k and grouped top-k
// gating, and SmallEP evaluates the gate locally before sorting tokens).
//
// Selection rule (DeepSeek-V3 gate): keys sel = s + bias; the E experts form
// n_group contiguous groups whose score is the sum of their two largest keys;
// the topk_group best groups are kept; the k largest keys among their
// experts are chosen, listed by decreasing key; equal values go to the lower
// index.  Weights: s[id_j] / sum_j s[id_j] * scaling, summed in slot order.
//
// Kernels:
//   router_logits_kernel (fewer than 256 tokens): 16 tokens x 256 experts per workgroup with the bf16
//     MFMA 16x16x32 (A = token rows, B = router rows, both read straight
//     from global memory as 16-byte pieces), over one of KS slices of K, so
//     that a few tokens still spread over enough workgroups; fp32 partial
//     logits [KS][T][E].
//   router_logits_tiled_kernel (256 tokens or more): 128 x 256 tiles through
//     LDS, also over K slices, the same partial layout.
//   router_select_kernel: one wave per token sums the KS partials in slice
//     order, applies the sigmoid and the bias, keeps the best groups, and
//     takes the k largest keys in k argmax rounds (k <= 16), or finds the
//     k-th largest key by a radix select over its bits and orders the k
//     chosen experts; lanes 0 .. k-1 write ids and weights.
#include "common.h"

#include <type_traits>

namespace moe {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kRouterMaxExperts = 1024; // one selection thread per expert
constexpr int kRouterMaxGroups = 64;
constexpr int kRouterMinChunk = 128;    // K elements per logits workgroup at least
constexpr int kArgmaxMaxK = 16;         // selection by k argmax rounds up to this k, a radix select beyond

__global__ __launch_bounds__(256) void router_logits_kernel(const uint16_t* __restrict__ x, int T, int H,
                                                            const uint16_t* __restrict__ w, int E, int kchunk,
                                                            float* __restrict__ part) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane & 15;   // A row (token) / B column (expert) this lane supplies
  const int kq = lane >> 4;  // K group: elements 8 kq .. 8 kq + 7 of each 32
  const int t0 = blockIdx.x * 16;
  const int e0 = blockIdx.y * 256 + wave * 64;
  const int ks = blockIdx.z;
  if (e0 >= E) return;  // the whole wave: no barrier in this kernel
  const int64_t k0 = (int64_t)ks * kchunk;
  // Rows beyond T or E read a valid row; their results are not stored.
  const uint16_t* xa = x + (int64_t)min(t0 + r, T - 1) * H + k0 + 8 * kq;
  const uint16_t* wb[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) wb[nt] = w + (int64_t)min(e0 + 16 * nt + r, E - 1) * H + k0 + 8 * kq;
  v4f acc[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) acc[nt] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int kk = 0; kk < kchunk; kk += 32) {
    const bf16x8 a = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(xa + kk));
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const bf16x8 b = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(wb[nt] + kk));
      acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[nt], 0, 0, 0);
    }
  }
  // Lane l holds logits of tokens t0 + 4 kq + i for expert e0 + 16 nt + r.
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = t0 + 4 * kq + i, e = e0 + 16 * nt + r;
      if (t < T && e < E) part[((int64_t)ks * T + t) * E + e] = acc[nt][i];
    }
}

// Many tokens: an LDS-tiled bf16 GEMM.  Workgroup = TM tokens x 256
// experts over one K slice, 512 threads; wave w computes tokens
// TM/2 (w / 4) + [0, TM/2) against experts 64 (w % 4) + [0, 64) (TM/8 MFMA
// 16x16x32 per 32-K step).  The 32-K tiles of both operands go through two
// LDS stages (each thread loads TM/8 bytes of x and 32 bytes of W_r per
// step); a 64-byte LDS row holds one row's 32 K values, which a quarter wave
// reads as 16 rows x 64 contiguous bytes.  The global loads run RING - 1
// steps ahead through a ring of registers (four slots for 128-token tiles,
// three for 256, which need twice the registers per slot): with one step of
// look-ahead the
// kernel was bound by the loads' latency (224.8 us at 32768 tokens, against
// 161.7 us with the ring).  Every tile reads the whole router weight (3.67 MB
// at the DeepSeek-V3 shape) from L2, so from 32768 tokens on, where 128-token
// tiles alone fill the chip, tiles of 256 tokens halve those reads (143.8
// against 161.7 us); below, the K slices that 256-token tiles need to fill
// the chip cost more than they save (8192 tokens: 43.8 against 43.0 us, and
// a slower selection over twice the slices).
constexpr int kRtN = 256, kRtK = 32;
constexpr int kRtBigTokens = 32768;  // 256-token tiles from here on
inline int router_tile_tokens(int64_t T) { return T >= kRtBigTokens ? 256 : 128; }

template <int TM, int RING>
__global__ __launch_bounds__(512) void router_logits_tiled_kernel(const uint16_t* __restrict__ x, int T, int H,
                                                                  const uint16_t* __restrict__ w, int E, int kchunk,
                                                                  float* __restrict__ part) {
  constexpr int XR = TM / 128;  // x rows per loader thread
  constexpr int WI = TM / 32;   // 16-token MFMA tiles per wave
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][TM * kRtK];
  __shared__ __attribute__((aligned(16))) uint16_t wsm[2][kRtN * kRtK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, kq = lane >> 4;
  const int wm = wave >> 2, wn = wave & 3;
  const int t0 = blockIdx.x * TM, e0 = blockIdx.y * kRtN, ks = blockIdx.z;
  const int64_t k0 = (int64_t)ks * kchunk;
  // Loader: thread tid moves x rows tid / 4 (+ 128) and W_r rows tid / 4 and
  // 128 + tid / 4 (16 bytes each at K 8 (tid % 4)); rows beyond T or E read
  // a valid row.
  const int lr = tid >> 2, lk = (tid & 3) * 8;
  const uint16_t* xg0 = x + (int64_t)min(t0 + lr, T - 1) * H + k0 + lk;
  const uint16_t* xg1 = x + (int64_t)min(t0 + (XR - 1) * 128 + lr, T - 1) * H + k0 + lk;
  const uint16_t* wg0 = w + (int64_t)min(e0 + lr, E - 1) * H + k0 + lk;
  const uint16_t* wg1 = w + (int64_t)min(e0 + 128 + lr, E - 1) * H + k0 + lk;
  v4f acc[WI][4];
#pragma unroll
  for (int i = 0; i < WI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
  const int nsteps = kchunk / kRtK;
  // Ring slot S holds step st's operands for st % kRtRing == S (steps past
  // the end reload the last one, so every step issues the same loads).
  uint4 rxa0, rxa1, rxa2, rxa3, rxb0, rxb1, rxb2, rxb3, rwa0, rwa1, rwa2, rwa3, rwb0, rwb1, rwb2, rwb3;
#define MOE_RT_LOAD(S, ST)                                                      \
  do {                                                                          \
    const int64_t o_ = (int64_t)min((ST), nsteps - 1) * kRtK;                   \
    rxa##S = *reinterpret_cast<const uint4*>(xg0 + o_);                         \
    if (XR > 1) rxb##S = *reinterpret_cast<const uint4*>(xg1 + o_);             \
    rwa##S = *reinterpret_cast<const uint4*>(wg0 + o_);                         \
    rwb##S = *reinterpret_cast<const uint4*>(wg1 + o_);                         \
  } while (0)
  // Step st in slot S: its operands into LDS stage st % 2, the barrier, the
  // loads of step st + RING - 1 into slot NEXT (stored one step ago), then
  // the step's MFMAs.  A stage is rewritten two steps after it was read,
  // behind the barrier of the step in between.
#define MOE_RT_STEP(S, NEXT, ST)                                                \
  do {                                                                          \
    const int st_ = (ST), b_ = st_ & 1;                                         \
    *reinterpret_cast<uint4*>(&xs[b_][lr * kRtK + lk]) = rxa##S;                \
    if (XR > 1) *reinterpret_cast<uint4*>(&xs[b_][(128 + lr) * kRtK + lk]) = rxb##S; \
    *reinterpret_cast<uint4*>(&wsm[b_][lr * kRtK + lk]) = rwa##S;               \
    *reinterpret_cast<uint4*>(&wsm[b_][(128 + lr) * kRtK + lk]) = rwb##S;       \
    __syncthreads();                                                            \
    MOE_RT_LOAD(NEXT, st_ + RING - 1);                                          \
    mma_stage(b_);                                                              \
  } while (0)
  auto mma_stage = [&](int b) {
    bf16x8 bb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      bb[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(&wsm[b][(64 * wn + 16 * j + r) * kRtK + 8 * kq]));
#pragma unroll
    for (int i = 0; i < WI; ++i) {
      const bf16x8 a = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const uint4*>(&xs[b][(TM / 2 * wm + 16 * i + r) * kRtK + 8 * kq]));
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bb[j], acc[i][j], 0, 0, 0);
    }
  };
  static_assert(RING == 3 || RING == 4, "the unrolled rings below have three or four slots");
  MOE_RT_LOAD(0, 0);
  MOE_RT_LOAD(1, 1);
  int st = 0;
  if constexpr (RING == 4) {
    MOE_RT_LOAD(2, 2);
    for (; st + 4 <= nsteps; st += 4) {
      MOE_RT_STEP(0, 3, st);
      MOE_RT_STEP(1, 0, st + 1);
      MOE_RT_STEP(2, 1, st + 2);
      MOE_RT_STEP(3, 2, st + 3);
    }
    if (st < nsteps) MOE_RT_STEP(0, 3, st);
    if (st + 1 < nsteps) MOE_RT_STEP(1, 0, st + 1);
    if (st + 2 < nsteps) MOE_RT_STEP(2, 1, st + 2);
  } else {
    for (; st + 3 <= nsteps; st += 3) {
      MOE_RT_STEP(0, 2, st);
      MOE_RT_STEP(1, 0, st + 1);
      MOE_RT_STEP(2, 1, st + 2);
    }
    if (st < nsteps) MOE_RT_STEP(0, 2, st);
    if (st + 1 < nsteps) MOE_RT_STEP(1, 0, st + 1);
  }
#undef MOE_RT_STEP
#undef MOE_RT_LOAD
  // Lane l holds logits of tokens (TM/2 wm + 16 i) + 4 kq + q for expert (64 wn + 16 j) + r.
#pragma unroll
  for (int i = 0; i < WI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = t0 + TM / 2 * wm + 16 * i + 4 * kq + q, e = e0 + 64 * wn + 16 * j + r;
        if (t < T && e < E) part[((int64_t)ks * T + t) * E + e] = acc[i][j][q];
      }
}

// (value, index) order of the selection: larger value first, then lower index.
__device__ __forceinline__ bool beats(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// The value of lane p(l) of a row of 16 lanes, for the DPP patterns below
// (a VALU operand modifier; no LDS traffic, unlike a shuffle).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
// Lane patterns that pair every lane with one of another part of its group,
// doubling the group each time: quads (lane ^ 1, lane ^ 2), then half rows
// (lane 7 - i of the 8) and rows (lane 15 - i of the 16).  A reduction that
// does not depend on the order of its operands gives every lane of a row the
// result over the row's 16 lanes.
constexpr int kDppQuadXor1 = 0xB1, kDppQuadXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

// Every lane gets the wave's largest (key, index) in the selection order.
__device__ __forceinline__ void wave_argmax(float& bk, int& be) {
  auto step = [&](float ok, int oe) {
    if (beats(ok, oe, bk, be)) {
      bk = ok;
      be = oe;
    }
  };
  step(dpp_f<kDppQuadXor1>(bk), dpp_i<kDppQuadXor1>(be));
  step(dpp_f<kDppQuadXor2>(bk), dpp_i<kDppQuadXor2>(be));
  step(dpp_f<kDppHalfMirror>(bk), dpp_i<kDppHalfMirror>(be));
  step(dpp_f<kDppMirror>(bk), dpp_i<kDppMirror>(be));
  // the four rows' results, as wave-uniform values
  float k0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, bk), 0));
  int e0 = __builtin_amdgcn_readlane(be, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) {
    const float kr = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, bk), 16 * r));
    const int er = __builtin_amdgcn_readlane(be, 16 * r);
    if (beats(kr, er, k0, e0)) {
      k0 = kr;
      e0 = er;
    }
  }
  bk = k0;
  be = e0;
}

// Selection: one wave per token (four tokens per 256-thread workgroup),
// lane l holding experts l, l + 64, ... (PER of them).  The KS partial
// logits are summed in slice order, then:
//   * group scores: for each group the two largest keys, by a wave
//     reduction of (largest, second) pairs; lane g ranks group g against
//     the others and the topk_group best are kept;
//   * k <= 16: k rounds of a wave argmax over (key, index), each taking the
//     largest remaining key, which gives the experts in slot order (k = 8:
//     8 rounds of 6 shuffle steps against 32 dependent radix steps plus an
//     ordering pass);
//   * larger k: the k-th largest kept key (in the (value, index) order) by a
//     radix select over the 32 bits of the keys mapped to ordered integers:
//     each bit costs PER ballots, with no per-expert comparisons against all
//     E; the k chosen experts (keys above the k-th, and the lowest indices of
//     those equal to it) are then ordered among themselves through LDS.
// ids / wts rows have k_out = k (+1 with a shared expert) columns.
__device__ __forceinline__ uint32_t ordered_bits(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// WIDE (few tokens, many K slices): one token per workgroup; the four waves
// each sum the slices q = w, w + 4, ... and wave 0 adds the four partial sums
// (in wave order) before it selects, so the slices are read in one round
// trip instead of several.
template <int PER, bool WIDE, int QB>
__global__ __launch_bounds__(256) void router_select_kernel(const float* __restrict__ part, int KS, int T, int E,
                                                            const float* __restrict__ bias, int k, int n_group,
                                                            int topk_group, float scaling, int shared,
                                                            int32_t* __restrict__ ids, float* __restrict__ wts) {
  __shared__ float sel_key[4][32], sel_s[4][32];
  __shared__ int sel_e[4][32];
  __shared__ float wide_sum[WIDE ? 3 : 1][WIDE ? 64 * PER : 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int slot = WIDE ? 0 : wave;
  const int64_t t = WIDE ? (int64_t)blockIdx.x : (int64_t)blockIdx.x * 4 + wave;
  if (t >= T) return;  // the whole wave (WIDE: the whole workgroup); no other barrier below
  const int epg = E / n_group;
  const int k_out = k + (shared >= 0 ? 1 : 0);

  // Logits: the KS slices summed in slice order; the loads of a batch of QB
  // slices go out together (slice index clamped, so every load is
  // unconditional).  QB follows the launch's slice count (2, 4, or 64 / PER
  // for more slices), so a launch with one or two slices does not issue the
  // loads of sixteen.
  float s[PER], key[PER];
  {
    float lg[PER], bv[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = min(lane + 64 * i, E - 1);
      bv[i] = bias ? bias[e] : 0.0f;
      lg[i] = 0.0f;
    }
    const int q_first = WIDE ? wave : 0, q_step = WIDE ? 4 : 1;
    for (int q0 = q_first; q0 < KS; q0 += QB * q_step) {
      float v[QB][PER];
#pragma unroll
      for (int q = 0; q < QB; ++q)
#pragma unroll
        for (int i = 0; i < PER; ++i)
          v[q][i] = part[((int64_t)min(q0 + q * q_step, KS - 1) * T + t) * E + min(lane + 64 * i, E - 1)];
#pragma unroll
      for (int q = 0; q < QB; ++q)
#pragma unroll
        for (int i = 0; i < PER; ++i)
          if (q0 + q * q_step < KS) lg[i] += v[q][i];
    }
    if constexpr (WIDE) {
      if (wave > 0) {
#pragma unroll
        for (int i = 0; i < PER; ++i) wide_sum[wave - 1][lane + 64 * i] = lg[i];
      }
      __syncthreads();
      if (wave > 0) return;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        lg[i] += wide_sum[0][lane + 64 * i];
        lg[i] += wide_sum[1][lane + 64 * i];
        lg[i] += wide_sum[2][lane + 64 * i];
      }
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      s[i] = 1.0f / (1.0f + expf(-lg[i]));
      key[i] = lane + 64 * i < E ? s[i] + bv[i] : -INFINITY;
    }
  }

  // Groups: score = sum of the two largest keys; lane g keeps group g's.
  if (n_group > 1) {
    float my_group = -INFINITY;
    if (epg <= 64 && 64 % epg == 0) {
      // Aligned groups (epg a power of two up to 64): register i holds groups
      // i * 64 / epg + (lane / epg); all are reduced at once inside their
      // epg-lane segments, then lane g fetches group g's score.
      float b1[PER], b2[PER];
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        b1[i] = key[i];
        b2[i] = -INFINITY;
      }
      // (largest, second) pairs merged with a partner lane of the segment:
      // within rows by DPP patterns (quads, half rows, rows), beyond by
      // shuffles.
      auto merge = [&](int i, float o1, float o2) {
        const float n2 = fmaxf(fminf(b1[i], o1), fmaxf(b2[i], o2));
        b1[i] = fmaxf(b1[i], o1);
        b2[i] = n2;
      };
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        if (epg > 1) merge(i, dpp_f<kDppQuadXor1>(b1[i]), dpp_f<kDppQuadXor1>(b2[i]));
        if (epg > 2) merge(i, dpp_f<kDppQuadXor2>(b1[i]), dpp_f<kDppQuadXor2>(b2[i]));
        if (epg > 4) merge(i, dpp_f<kDppHalfMirror>(b1[i]), dpp_f<kDppHalfMirror>(b2[i]));
        if (epg > 8) merge(i, dpp_f<kDppMirror>(b1[i]), dpp_f<kDppMirror>(b2[i]));
        for (int m = 16; m < epg; m <<= 1) merge(i, __shfl_xor(b1[i], m), __shfl_xor(b2[i], m));
      }
      const int gpr = 64 / epg;  // groups per register
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const float v = __shfl(b1[i] + b2[i], (lane % gpr) * epg);
        if (lane / gpr == i) my_group = v;
      }
    } else {
      for (int g = 0; g < n_group; ++g) {
        float b1 = -INFINITY, b2 = -INFINITY;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
          const int e = lane + 64 * i;
          if (e < E && e / epg == g) {
            const float v = key[i];
            if (v > b1) {
              b2 = b1;
              b1 = v;
            } else if (v > b2) {
              b2 = v;
            }
          }
        }
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) {
          const float o1 = __shfl_xor(b1, m), o2 = __shfl_xor(b2, m);
          const float n2 = fmaxf(fminf(b1, o1), fmaxf(b2, o2));
          b1 = fmaxf(b1, o1);
          b2 = n2;
        }
        if (lane == g) my_group = b1 + b2;
      }
    }
    int rank = 0;
    for (int h = 0; h < n_group; ++h) {
      const float gh = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, my_group), h));
      rank += beats(gh, h, my_group, lane) ? 1 : 0;
    }
    const unsigned long long kept_groups = __ballot(lane < n_group && rank < topk_group);  // bit g: group g kept
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = lane + 64 * i;
      if (!((kept_groups >> (e < E ? e / epg : 0)) & 1ull)) key[i] = -INFINITY;
    }
  }

  if (k <= kArgmaxMaxK) {
    // Small k: k rounds of a wave argmax over (key, expert index), each round
    // taking the largest remaining key (the lower index on equal keys), so
    // the experts come out in slot order (decreasing key) with no ordering
    // step; lane j keeps slot j's expert and sigmoid score.
    int my_e = 0;
    float my_s = 0.0f;
    for (int j = 0; j < k; ++j) {
      float bk = key[0];
      int be = lane;
#pragma unroll
      for (int i = 1; i < PER; ++i)
        if (key[i] > bk) {  // registers hold increasing indices: ties keep the lower one
          bk = key[i];
          be = lane + 64 * i;
        }
      wave_argmax(bk, be);  // every lane ends with the same best
      float sv = s[0];
#pragma unroll
      for (int i = 1; i < PER; ++i)
        if ((be >> 6) == i) sv = s[i];
      sv = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sv), be & 63));
      if (lane == j) {
        my_e = be;
        my_s = sv;
      }
#pragma unroll
      for (int i = 0; i < PER; ++i)
        if (lane + 64 * i == be) key[i] = -INFINITY;
    }
    if (lane < k) {
      ids[t * k_out + lane] = my_e;
      sel_s[slot][lane] = my_s;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < k) {
      float total = 0.0f;
      for (int j = 0; j < k; ++j) total += sel_s[slot][j];
      wts[t * k_out + lane] = (my_s / total) * scaling;
    }
    if (shared >= 0 && lane == 0) {
      ids[t * k_out + k] = shared;
      wts[t * k_out + k] = 1.0f;
    }
    return;
  }

  // Radix select of the k-th largest key: prefix of the ordered bits, and
  // `need` = how many of the keys equal to it are chosen (lowest index first).
  uint32_t u[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) u[i] = ordered_bits(key[i]);
  uint32_t prefix = 0, mask = 0;
  int need = k;
  for (int b = 31; b >= 0; --b) {
    const uint32_t bit = 1u << b;
    int c1 = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) c1 += __popcll(__ballot((u[i] & mask) == prefix && (u[i] & bit)));
    if (c1 >= need) prefix |= bit;
    else need -= c1;
    mask |= bit;
  }
  // Chosen: u > prefix, or u == prefix and among the first `need` such keys
  // in expert order (e = lane + 64 i: register i, then lane).
  const unsigned long long below = (1ull << lane) - 1ull;
  int eq_before = 0, n_sel = 0;
  bool chosen[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const unsigned long long eq = __ballot(u[i] == prefix);
    const int my_eq = eq_before + __popcll(eq & below);
    chosen[i] = u[i] > prefix || (u[i] == prefix && my_eq < need);
    eq_before += __popcll(eq);
  }
  // Compact the k chosen (expert order) into LDS, then each takes its rank.
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const unsigned long long cb = __ballot(chosen[i]);
    if (chosen[i]) {
      const int at = n_sel + __popcll(cb & below);
      sel_key[slot][at] = key[i];
      sel_s[slot][at] = s[i];
      sel_e[slot][at] = lane + 64 * i;
    }
    n_sel += __popcll(cb);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  float cs = 0.0f;
  int ce = 0, crank = 0;
  if (lane < k) {
    const float kv = sel_key[slot][lane];
    ce = sel_e[slot][lane];
    cs = sel_s[slot][lane];
    for (int j = 0; j < k; ++j) crank += beats(sel_key[slot][j], sel_e[slot][j], kv, ce) ? 1 : 0;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (lane < k) {
    ids[t * k_out + crank] = ce;
    sel_s[slot][crank] = cs;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (lane < k) {
    float total = 0.0f;
    for (int j = 0; j < k; ++j) total += sel_s[slot][j];
    wts[t * k_out + lane] = (sel_s[slot][lane] / total) * scaling;
  }
  if (shared >= 0 && lane == 0) {
    ids[t * k_out + k] = shared;
    wts[t * k_out + k] = 1.0f;
  }
}

// From this many tokens on the logits use the tiled kernel.
constexpr int kRouterTiledMinTokens = 256;

// K slices of the logits: enough workgroups to cover the chip (256 or
// more), each slice a divisor of H / 32 slices of 32 and at least
// kRouterMinChunk elements.
int router_slices(int32_t T, int32_t H, int32_t E) {
  const bool tiled = T >= kRouterTiledMinTokens;
  const int tm = router_tile_tokens(T);
  const int64_t tiles = tiled ? ((int64_t)T + tm - 1) / tm * (((int64_t)E + kRtN - 1) / kRtN)
                              : ((int64_t)T + 15) / 16 * (((int64_t)E + 255) / 256);
  const int64_t want = tiles >= 256 ? 1 : (256 + tiles - 1) / tiles;
  const int n32 = H / 32;
  int best = 1;
  for (int ks = 1; ks <= n32; ++ks)
    if (n32 % ks == 0 && (int64_t)ks <= want && (H / ks) >= kRouterMinChunk) best = ks;
  return best;
}

}  // namespace

}  // namespace moe

using namespace moe;

extern "C" size_t moe_router_workspace(int32_t T, int32_t H, int32_t E) {
  if (T <= 0 || H <= 0 || E <= 0 || H % 32) return 0;
  return (size_t)router_slices(T, H, E) * (size_t)T * (size_t)E * sizeof(float);
}

extern "C" moe_status_t moe_router(const uint16_t* x_bf16, int32_t T, int32_t H, const uint16_t* w_router_bf16,
                                   const float* bias, int32_t E, int32_t k, moe_router_cfg_t cfg,
                                   int32_t* topk_ids, float* topk_w, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  if (T < 0 || H <= 0 || H % 32 || E < 1 || E > kRouterMaxExperts)
    return fail(MOE_ERR_INVALID_ARG, "moe_router: T=%d H=%d E=%d (need H %% 32 == 0, 1 <= E <= %d)", T, H, E,
                kRouterMaxExperts);
  if (cfg.n_group < 1 || cfg.n_group > kRouterMaxGroups || E % cfg.n_group || (cfg.n_group > 1 && E / cfg.n_group < 2) ||
      cfg.topk_group < 1 || cfg.topk_group > cfg.n_group || k < 1 || k > 32 ||
      k > cfg.topk_group * (E / cfg.n_group))
    return fail(MOE_ERR_INVALID_ARG, "moe_router: k=%d n_group=%d topk_group=%d for E=%d", k, cfg.n_group,
                cfg.topk_group, E);
  if (!(cfg.routed_scaling > 0.0f)) return fail(MOE_ERR_INVALID_ARG, "moe_router: routed_scaling must be > 0");
  if (cfg.shared_expert >= 0 && k > 31) return fail(MOE_ERR_INVALID_ARG, "moe_router: k + 1 slots exceed 32");
  if (T == 0) return MOE_OK;
  if (!x_bf16 || !w_router_bf16 || !topk_ids || !topk_w) return fail(MOE_ERR_INVALID_ARG, "moe_router: null pointer");
  if (!aligned(x_bf16, 16) || !aligned(w_router_bf16, 16))
    return fail(MOE_ERR_INVALID_ARG, "moe_router: x and the router weight must be 16-byte aligned");
  const size_t need = moe_router_workspace(T, H, E);
  if (!ws || ws_bytes < need) return fail(MOE_ERR_WORKSPACE, "moe_router: workspace %zu bytes < %zu", ws_bytes, need);
  if (!aligned(ws, 4)) return fail(MOE_ERR_INVALID_ARG, "moe_router: misaligned workspace");
  const int ks = router_slices(T, H, E);
  float* part = static_cast<float*>(ws);
  if (T >= kRouterTiledMinTokens) {
    const int tm = router_tile_tokens(T);
    const dim3 grid((unsigned)((T + tm - 1) / tm), (unsigned)((E + kRtN - 1) / kRtN), (unsigned)ks);
    if (tm == 256)
      MOE_LAUNCH("router_logits", (router_logits_tiled_kernel<256, 3>), grid, dim3(512), 0, stream, x_bf16, T, H,
                 w_router_bf16, E, H / ks, part);
    else
      MOE_LAUNCH("router_logits", (router_logits_tiled_kernel<128, 4>), grid, dim3(512), 0, stream, x_bf16, T, H,
                 w_router_bf16, E, H / ks, part);
  } else {
    const dim3 grid((unsigned)((T + 15) / 16), (unsigned)((E + 255) / 256), (unsigned)ks);
    MOE_LAUNCH("router_logits", router_logits_kernel, grid, dim3(256), 0, stream, x_bf16, T, H, w_router_bf16, E,
               H / ks, part);
  }
  moe_status_t st = check_launch("moe_router");
  if (st != MOE_OK) return st;
  // Few tokens with many K slices: one token per workgroup (WIDE).
  const bool wide = ks >= 8 && T <= 64;
  const dim3 sgrid((unsigned)(wide ? T : (T + 3) / 4)), sblock(256);
#define MOE_ROUTER_SELECT_Q(P, W, Q)                                                                               \
  MOE_LAUNCH("router_select", (router_select_kernel<P, W, Q>), sgrid, sblock, 0, stream, part, ks, T, E, bias, k,    \
             cfg.n_group, cfg.topk_group, cfg.routed_scaling, cfg.shared_expert, topk_ids, topk_w)
#define MOE_ROUTER_SELECT(P)                                                                                       \
  do {                                                                                                             \
    constexpr int qb_ = (64 / (P)) > 1 ? 64 / (P) : 1;                                                             \
    if (wide) MOE_ROUTER_SELECT_Q(P, true, qb_);                                                                   \
    else if (ks <= 2) MOE_ROUTER_SELECT_Q(P, false, 2);                                                            \
    else if (ks <= 4) MOE_ROUTER_SELECT_Q(P, false, 4);                                                            \
    else MOE_ROUTER_SELECT_Q(P, false, qb_);                                                                       \
  } while (0)
  const int per = (E + 63) / 64;
  if (per <= 1) MOE_ROUTER_SELECT(1);
  else if (per <= 2) MOE_ROUTER_SELECT(2);
  else if (per <= 4) MOE_ROUTER_SELECT(4);
  else if (per <= 8) MOE_ROUTER_SELECT(8);
  else MOE_ROUTER_SELECT(16);
#undef MOE_ROUTER_SELECT
#undef MOE_ROUTER_SELECT_Q
  return check_launch("moe_router");
}
