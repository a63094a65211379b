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
// Two kernels:
//   router_logits_kernel: 16 tokens x 256 experts per workgroup with the bf16
//     MFMA 16x16x32 (A = token rows, B = router rows, both read straight
//     from global memory as 16-byte pieces), over one of KS slices of K, so
//     that a few tokens still spread over enough workgroups; fp32 partial
//     logits [KS][T][E].
//   router_select_kernel: one wave per token sums the KS partials in slice
//     order, applies the sigmoid and the bias, ranks groups and experts with
//     wave shuffles and writes ids and weights.
#include "common.h"

namespace moe {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kRouterMaxPerLane = 16;   // experts per lane in the selection (E <= 1024)
constexpr int kRouterMaxGroups = 64;    // one group score per lane
constexpr int kRouterMinChunk = 128;    // K elements per logits workgroup at least

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

// (value, index) order of the selection: larger value first, then lower index.
__device__ __forceinline__ bool beats(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// ids / wts rows have k_out = k (+1 with a shared expert) columns.  PER:
// experts per lane (lane l holds experts l*PER .. l*PER + PER - 1).
template <int PER>
__global__ __launch_bounds__(256) void router_select_kernel(const float* __restrict__ part, int KS, int T, int E,
                                                            const float* __restrict__ bias, int k, int n_group,
                                                            int topk_group, float scaling, int shared,
                                                            int32_t* __restrict__ ids, float* __restrict__ wts) {
  const int k_out = k + (shared >= 0 ? 1 : 0);
  __shared__ float chosen[4][32];  // the chosen experts' scores of each wave's token
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // the whole wave
  constexpr int per = PER;
  const int epg = E / n_group;
  // Logits: the KS slices summed in slice order; QB slices of all the lane's
  // experts are loaded before any is added (a few tokens have many slices).
  constexpr int QB = 128 / PER;
  float lg[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) lg[i] = 0.0f;
  for (int q0 = 0; q0 < KS; q0 += QB) {
    float v[QB][PER];
#pragma unroll
    for (int q = 0; q < QB; ++q)
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int e = lane * PER + i;
        v[q][i] = (q0 + q < KS && e < E) ? part[((int64_t)(q0 + q) * T + t) * E + e] : 0.0f;
      }
#pragma unroll
    for (int q = 0; q < QB; ++q)
#pragma unroll
      for (int i = 0; i < PER; ++i)
        if (q0 + q < KS) lg[i] += v[q][i];
  }
  float s[kRouterMaxPerLane], key[kRouterMaxPerLane];
#pragma unroll
  for (int i = 0; i < kRouterMaxPerLane; ++i) {
    const int e = lane * per + i;
    s[i] = 0.0f;
    key[i] = -INFINITY;
    if (i < per && e < E) {
      s[i] = 1.0f / (1.0f + expf(-lg[i]));
      key[i] = s[i] + (bias ? bias[e] : 0.0f);
    }
  }
  // Group scores: the two largest keys of group g over the wave (values only,
  // merged pairwise), kept by lane g.
  float my_group = -INFINITY;
  for (int g = 0; g < n_group; ++g) {
    float b1 = -INFINITY, b2 = -INFINITY;
#pragma unroll
    for (int i = 0; i < kRouterMaxPerLane; ++i) {
      const int e = lane * per + i;
      if (i < per && e < E && e / epg == g) {
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
    const float score = n_group > 1 ? b1 + b2 : 0.0f;  // one group: all experts are kept anyway
    if (lane == g) my_group = score;
  }
  int rank = 0;
  for (int h = 0; h < n_group; ++h) {
    const float gh = __shfl(my_group, h);
    rank += beats(gh, h, my_group, lane) ? 1 : 0;
  }
  const int kept_group = (lane < n_group && rank < topk_group) ? 1 : 0;
#pragma unroll
  for (int i = 0; i < kRouterMaxPerLane; ++i) {
    const int e = lane * per + i;
    const int kept = __shfl(kept_group, (i < per && e < E) ? e / epg : 0);
    if (!(i < per && e < E) || !kept) key[i] = -INFINITY;
  }
  // k rounds of a wave-wide arg-max over (key, index), carrying the score.
  float total = 0.0f;
  for (int j = 0; j < k; ++j) {
    float bv = -INFINITY, bs = 0.0f;
    int bi = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < kRouterMaxPerLane; ++i) {
      const int e = lane * per + i;
      if (i < per && e < E && beats(key[i], e, bv, bi)) {
        bv = key[i];
        bi = e;
        bs = s[i];
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float ov = __shfl_xor(bv, m), os = __shfl_xor(bs, m);
      const int oi = __shfl_xor(bi, m);
      if (beats(ov, oi, bv, bi)) {
        bv = ov;
        bi = oi;
        bs = os;
      }
    }
#pragma unroll
    for (int i = 0; i < kRouterMaxPerLane; ++i)
      if (lane * per + i == bi) key[i] = -INFINITY;
    total += bs;
    if (lane == 0) {
      ids[(int64_t)t * k_out + j] = bi;
      chosen[threadIdx.x >> 6][j] = bs;
    }
  }
  if (lane == 0) {
    for (int j = 0; j < k; ++j) wts[(int64_t)t * k_out + j] = (chosen[threadIdx.x >> 6][j] / total) * scaling;
    if (shared >= 0) {
      ids[(int64_t)t * k_out + k] = shared;
      wts[(int64_t)t * k_out + k] = 1.0f;
    }
  }
}

// K slices of the logits: enough workgroups for a few tokens, each slice at
// least kRouterMinChunk elements and a divisor of H / 32 slices of 32.
int router_slices(int32_t T, int32_t H, int32_t E) {
  const int64_t tiles = ((int64_t)T + 15) / 16 * (((int64_t)E + 255) / 256);
  const int64_t want = tiles >= 256 ? 1 : 256 / tiles;
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
  if (T < 0 || H <= 0 || H % 32 || E < 1 || E > 64 * kRouterMaxPerLane)
    return fail(MOE_ERR_INVALID_ARG, "moe_router: T=%d H=%d E=%d (need H %% 32 == 0, 1 <= E <= %d)", T, H, E,
                64 * kRouterMaxPerLane);
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
  const dim3 grid((unsigned)((T + 15) / 16), (unsigned)((E + 255) / 256), (unsigned)ks);
  MOE_LAUNCH("router_logits", router_logits_kernel, grid, dim3(256), 0, stream, x_bf16, T, H, w_router_bf16, E, H / ks,
             part);
  moe_status_t st = check_launch("moe_router");
  if (st != MOE_OK) return st;
  const int per = (E + 63) / 64;
  const dim3 sgrid((unsigned)((T + 3) / 4));
#define MOE_ROUTER_SELECT(P)                                                                                  \
  MOE_LAUNCH("router_select", router_select_kernel<P>, sgrid, dim3(256), 0, stream, part, ks, T, E, bias, k,  \
             cfg.n_group, cfg.topk_group, cfg.routed_scaling, cfg.shared_expert, topk_ids, topk_w)
  if (per <= 1) MOE_ROUTER_SELECT(1);
  else if (per <= 2) MOE_ROUTER_SELECT(2);
  else if (per <= 4) MOE_ROUTER_SELECT(4);
  else if (per <= 8) MOE_ROUTER_SELECT(8);
  else MOE_ROUTER_SELECT(16);
#undef MOE_ROUTER_SELECT
  return check_launch("moe_router");
}
