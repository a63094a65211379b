// Decode down projection fused with the router-weighted combine, for small
// batches (R = T * k expert rows in all, R <= kDcMaxRows, K = I <= kDcMaxK).
//
// One workgroup owns 16 NT output columns [n0, n0 + 16 NT) of the layer and
// computes them for every active expert, so the expert rows of the whole
// batch never leave the workgroup: it combines them per token in LDS and
// writes only the bf16 layer output (the fp32 expert rows are not written).
// No workgroup depends on another.
//
// Per expert the arithmetic is the decode down kernel's (Fine-grained CPU
// Parallelism: down after SiLU(gate) * up; FP8 Block Scaling Format):
//   * h rows quantized per row per 128 (as moe_quant_rows_f32) into LDS;
//   * one FP8 MFMA 16x16x128 per 128-K block (A: the expert's token rows,
//     B: 16 W_down rows), promoted as acc += d * (sh[row, b] * s_down[n/128, b]);
//   * the K blocks split over four waves as kw, kw + 4, kw + 8, ... and the
//     four partials summed in wave order;
// and the combine is the definition's order (combine8_of).  The output is
// therefore bit-identical to the decode down kernel followed by moe_combine.
//
// Waves: WAVES = (expert slot s = wave / 4) x (K part kw = wave % 4); wave
// (s, kw) takes experts s, s + WAVES / 4, ... and streams their K blocks kw,
// kw + 4, ... as one list of items through a window of W items in registers,
// with no barrier inside the loop.  At the end of each expert it stores the
// expert's rows of its partial sum in LDS by expert row; after one barrier
// the four partials of each row are summed in wave order.
#include "common.h"

namespace moe {

namespace {

constexpr int kDcMaxRows = 16;                // R = T * k (beyond, H / 16 workgroups stream too few bytes per CU)
constexpr int kDcMaxTokens = 16;              // rows of one expert: one 16-row MFMA operand
constexpr int kDcMaxK = 2048;                 // I
constexpr int kDcMaxExperts = 1024;          // four 256-expert chunks of offsets

struct DownCombineArgs {
  const float* h;           // fp32 [R, K]: SiLU(G) * U rows in expert-sorted order
  const int32_t* offsets;   // [E+1]
  int E;
  const uint8_t* w;         // W_down [E, N, K], packed tiles
  const float* s;           // [E, N/128, K/128]
  int N, K;
  const int32_t* dest_row;  // [T * k]
  const float* topk_w;      // [T * k]
  int topk, tokens;
  uint16_t* out;            // bf16 [T, N]
  const int32_t* ids;       // SLOT1 (T = 1): the token's expert ids; h row j is slot j (offsets, dest_row unused)
};

// The active experts (those with rows) of slot `sub`: the a-th active
// expert in expert order with a = sub + SLOTS g goes to lane g as (expert, first
// row, row count); other lanes hold zeros.  Returns the number of active
// experts.  NCH chunks of 256 experts cover E; all their offsets are loaded
// first (addresses clamped to E, no branch), so the lookup costs one L2
// latency before the weight stream can start.
template <int NCH, int SLOTS>
__device__ __forceinline__ int active_experts(const int32_t* __restrict__ offsets, int E, int sub, int& v_e,
                                              int& v_p0, int& v_m) {
  const int lane = threadIdx.x & 63;
  int o[NCH][5];
#pragma unroll
  for (int q = 0; q < NCH; ++q) {
#pragma unroll
    for (int c = 0; c < 4; ++c) o[q][c] = offsets[min(256 * q + 64 * c + lane, E)];
    o[q][4] = offsets[min(256 * q + 256 + lane, E)];  // lane 0's: the end of the chunk
  }
  int n_act = 0, found = 0;
  v_e = 0;
  v_p0 = 0;
  v_m = 0;
#pragma unroll
  for (int q = 0; q < NCH; ++q) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int x = 256 * q + 64 * c + lane;
      const int nxt_first = __shfl(o[q][c + 1], 0);
      const int up = __shfl_down(o[q][c], 1);
      const int nxt = lane < 63 ? up : nxt_first;
      const bool on = x < E && nxt > o[q][c];
      const unsigned long long bal = __ballot(on);
      const int rank =
          n_act + (int)__builtin_amdgcn_mbcnt_hi((unsigned)(bal >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)bal, 0u));
      // this slot's experts in this chunk, in increasing order = increasing g
      unsigned long long want = __ballot(on && rank >= sub && ((rank - sub) & (SLOTS - 1)) == 0);
      while (want != 0ull && found < 64) {
        const int pos = __ffsll((long long)want) - 1;
        const int p0 = __builtin_amdgcn_readlane(o[q][c], pos);
        const int m = __builtin_amdgcn_readlane(nxt, pos) - p0;
        if (lane == found) {
          v_e = 256 * q + 64 * c + pos;
          v_p0 = p0;
          v_m = m;
        }
        ++found;
        want &= want - 1ull;
      }
      n_act += __popcll(bal);
    }
  }
  return n_act;
}

// One token (SLOT1): the same lanes as active_experts, from the token's ids
// in slot order: slot j is expert ids[j] with one row, row j, when the id
// lies in [0, E) and no earlier slot has it (the slots the sort keeps).
// Returns the number of such slots.
template <int SLOTS>
__device__ __forceinline__ int active_slots(const int32_t* __restrict__ ids, int k, int E, int sub, int& v_e,
                                            int& v_p0, int& v_m) {
  const int lane = threadIdx.x & 63;
  const int idv = lane < k ? ids[lane] : -1;
  bool dup = false;
  for (int i = 0; i < k; ++i) {
    const int o = __shfl(idv, i);
    dup |= i < lane && o == idv;
  }
  const bool on = lane < k && idv >= 0 && idv < E && !dup;
  const unsigned long long bal = __ballot(on);
  const int rank = (int)__builtin_amdgcn_mbcnt_hi((unsigned)(bal >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)bal, 0u));
  unsigned long long want = __ballot(on && rank >= sub && ((rank - sub) & (SLOTS - 1)) == 0);
  v_e = 0;
  v_p0 = 0;
  v_m = 0;
  int found = 0;
  while (want != 0ull) {
    const int pos = __ffsll((long long)want) - 1;
    const int e = __builtin_amdgcn_readlane(idv, pos);
    if (lane == found) {
      v_e = e;
      v_p0 = pos;
      v_m = 1;
    }
    ++found;
    want &= want - 1ull;
  }
  return __popcll(bal);
}

// NT: 16-column operands per workgroup; HQ: h row blocks per 16-lane group
// loaded before the weight window (the rest, if R * K / 128 > 64 HQ, are
// loaded after it); W: items in the weight window; NCH: 256-expert chunks
// of the offsets (E <= 256 NCH); WAVES: 4 K parts x WAVES / 4 expert slots;
// SLOT1: one token, experts from p.ids in slot order (active_slots).
template <int NT, int HQ, int W, int NCH, int WAVES, bool SLOT1 = false>
__global__ __launch_bounds__(64 * WAVES) void ffn_decode_down_combine_kernel(DownCombineArgs p) {
  constexpr int kCols = 16 * NT;
  constexpr int kDcThreads = 64 * WAVES;
  constexpr int kSlots = WAVES / 4;
  static_assert(kSlots == 1 || kSlots == 2 || kSlots == 4, "expert slots: a power of two");
  __shared__ __attribute__((aligned(16))) uint8_t qh[kDcMaxRows * kDcMaxK];
  __shared__ float sh[kDcMaxRows * (kDcMaxK / kBlock)];
  __shared__ float part[4 * kDcMaxRows * kCols];  // [K part][expert row][column]
  __shared__ __attribute__((aligned(16))) float yl[kDcMaxRows * kCols];
  __shared__ int32_t dest_id[SLOT1 ? kDcMaxRows : 1];  // SLOT1: slot j's row is row j

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int sub = wave >> 2, kw = wave & 3;
  const int r = lane & 15, kq = lane >> 4;
  const int nb = p.K / kBlock;
  const int R = p.tokens * p.topk;
  const int n0 = blockIdx.x * kCols;

  // This thread's first HQ h row blocks (g = tid/16, tid/16 + 64, ...) go
  // out first; they are quantized once the weight loads are in flight.
  // Blocks past the last one load the last one again (not quantized), so
  // the loads are not behind a branch whose join would wait for them.
  constexpr int kHq = HQ;
  float hv[kHq][8];
#pragma unroll
  for (int q = 0; q < kHq; ++q) {
    const int g = min((tid >> 4) + q * (kDcThreads / 16), R * nb - 1);
    const int row = g / nb, b = g - row * nb;
    load8_f32(p.h + (int64_t)row * p.K + b * kBlock + (tid & 15) * 8, hv[q]);
  }

  // Active experts, found by every wave on its own (no barrier): lane g
  // receives expert a = sub + kSlots g, the a-th expert with rows (expert
  // order), with its first row and row count.
  int v_e, v_p0, v_m;
  const int n_act = SLOT1 ? active_slots<kSlots>(p.ids, p.topk, p.E, sub, v_e, v_p0, v_m)
                          : active_experts<NCH, kSlots>(p.offsets, p.E, sub, v_e, v_p0, v_m);

  // Items of this wave: (expert a = sub + kSlots g, block j) for g < n_mine, j < nkw.
  const int nkw = (nb - kw + 3) / 4;
  const int n_mine = n_act > sub ? (n_act - sub + kSlots - 1) / kSlots : 0;
  const int n_items = n_mine * nkw;
  auto uni = [](int v, int l) { return __builtin_amdgcn_readlane(v, l); };
  // Lane i: the weight scale of item i, read by readlane at item i (its
  // load is issued before the weight window and waited for with it).
  float wsv;
  {
    const int g = lane / max(nkw, 1), j = lane - g * max(nkw, 1);
    const int e_g = __shfl(v_e, min(g, 63));
    wsv = lane < n_items ? p.s[((int64_t)e_g * (p.N / kBlock) + n0 / kBlock) * nb + kw + 4 * j] : 0.0f;
  }
  v8i wbuf[W][NT];
  // Item it (clamped into the list; a wave without items loads expert 0's
  // first block, which is never used).
  auto load_item = [&](int it, v8i (&w)[NT]) {
    const int g = it / max(nkw, 1), j = it - g * max(nkw, 1);
    const int e = n_items > 0 ? uni(v_e, g) : 0;
    const int bk = min(kw + 4 * j, nb - 1);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      w[nt] = load_v8i_packed(p.w + (((int64_t)e * p.N + n0 + 16 * nt) / 16 * nb + bk) * kTileBytes +
                              packed_lane_offset(0, kq, r));
  };
  // The window is refilled with the same number of loads on every item
  // (past the end: the last item again), so the wait before each item's
  // MFMA is a fixed count that leaves the later items' loads in flight.
#pragma unroll
  for (int u = 0; u < W; ++u) load_item(min(u, max(n_items - 1, 0)), wbuf[u]);

  // h quantized per 128 into LDS (16 lanes per row block).
  auto quant_block = [&](int g, const float (&v)[8]) {
    const int row = g / nb, b = g - row * nb, q16 = tid & 15;
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[i]));
#pragma unroll
    for (int m = 8; m >= 1; m >>= 1) amax = fmaxf(amax, __shfl_xor(amax, m, 16));
    const float sc = amax / kE4M3Max;
    const uint32_t lo = quantize4_e4m3(v[0], v[1], v[2], v[3], sc);
    const uint32_t hi = quantize4_e4m3(v[4], v[5], v[6], v[7], sc);
    *reinterpret_cast<uint2*>(qh + row * p.K + b * kBlock + q16 * 8) = make_uint2(lo, hi);
    if (q16 == 0) sh[row * nb + b] = sc;
  };
#pragma unroll
  for (int q = 0; q < kHq; ++q) {
    const int g = (tid >> 4) + q * (kDcThreads / 16);
    if (g < R * nb) quant_block(g, hv[q]);  // whole 16-lane groups
  }
  for (int g = (tid >> 4) + kHq * (kDcThreads / 16); g < R * nb; g += kDcThreads / 16) {
    float v[8];
    load8_f32(p.h + (int64_t)(g / nb) * p.K + (g - (g / nb) * nb) * kBlock + (tid & 15) * 8, v);
    quant_block(g, v);
  }
  // Partials start at zero: a wave without K blocks (K < 512) adds +0.0, as
  // the decode down kernel's does.
  for (int i = tid; i < 4 * kDcMaxRows * kCols; i += kDcThreads) part[i] = 0.0f;
  if (SLOT1 && tid < kDcMaxRows) dest_id[tid] = tid;
  __syncthreads();

  v4f acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = v4f{0.f, 0.f, 0.f, 0.f};
  for (int it0 = 0; it0 < n_items; it0 += W) {
#pragma unroll
    for (int u = 0; u < W; ++u) {
      const int it = it0 + u;
      if (it < n_items) {
        const int g = it / nkw, j = it - g * nkw;
        const int p0 = uni(v_p0, g), m = uni(v_m, g);
        const int bk = kw + 4 * j;
        const float ws = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wsv), it));
        // A rows beyond the expert's m rows read a valid row; their outputs are never kept.
        const v8i afrag = load_v8i_ksplit(qh + (p0 + min(r, m - 1)) * p.K + bk * kBlock + kq * 16);
        float sa[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = 4 * kq + i;
          sa[i] = row < m ? sh[(p0 + row) * nb + bk] : 0.0f;
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const v4f d = mfma_f8_16x16x128(afrag, wbuf[u][nt]);
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[nt][i] += d[i] * (sa[i] * ws);
        }
        if (j == nkw - 1) {  // the expert's last block: keep its rows, restart
          float* dst = part + kw * kDcMaxRows * kCols;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int row = 4 * kq + i;  // MFMA output: lane holds rows 4 kq + i, column r
              if (row < m) dst[(p0 + row) * kCols + nt * 16 + r] = acc[nt][i];
              acc[nt][i] = 0.0f;
            }
        }
      }
      load_item(min(it + W, n_items - 1), wbuf[u]);
    }
  }
  __syncthreads();
  // Rows of the active experts: the four K parts summed in wave order.
  for (int i = tid; i < R * kCols; i += kDcThreads) {
    float v = part[i];
    v += part[kDcMaxRows * kCols + i];
    v += part[2 * kDcMaxRows * kCols + i];
    v += part[3 * kDcMaxRows * kCols + i];
    yl[i] = v;
  }
  __syncthreads();

  // Combine: 8 columns per thread.
  constexpr int kPerTok = kCols / 8;
  for (int idx = tid; idx < p.tokens * kPerTok; idx += kDcThreads) {
    const int t = idx / kPerTok;
    const int c = (idx - t * kPerTok) * 8;
    *reinterpret_cast<uint4*>(p.out + (int64_t)t * p.N + n0 + c) =
        combine8_of([&](int64_t row) { return yl + row * kCols + c; }, SLOT1 ? dest_id : p.dest_row, p.topk_w,
                    p.topk, t);
  }
}

}  // namespace

// True when the fused down + combine takes this batch.
bool decode_down_combine_fits(const moe_dims_t& d, int32_t T) {
  return T >= 1 && T <= kDcMaxTokens && (int64_t)T * d.topk <= kDcMaxRows && d.inter <= kDcMaxK &&
         d.n_experts <= kDcMaxExperts && d.hidden % 32 == 0;
}

// y = down(h) of every active expert combined per token into out (bf16 [T, H]).
moe_status_t run_ffn_decode_down_combine(const moe_dims_t& d, int32_t T, const float* h, const int32_t* offsets,
                                         const uint8_t* w_down, const float* s_down, const int32_t* dest_row,
                                         const float* topk_w, uint16_t* out, hipStream_t stream) {
  if (!decode_down_combine_fits(d, T))
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "decode down+combine: T=%d (max %d), T*k=%d (max %d), I=%d (max %d)", T,
                kDcMaxTokens, T * d.topk, kDcMaxRows, d.inter, kDcMaxK);
  DownCombineArgs a{};
  a.h = h; a.offsets = offsets; a.E = d.n_experts;
  a.w = w_down; a.s = s_down; a.N = d.hidden; a.K = d.inter;
  a.dest_row = dest_row; a.topk_w = topk_w; a.topk = d.topk; a.tokens = T; a.out = out;
  // 16 columns and 8 waves (two expert slots x four K parts) per workgroup:
  // two workgroups fit on a CU (94 VGPRs, 39 KB of LDS), so all H / 16 of
  // them are resident at once on all CUs (at H = 7168: 448 on 256 CUs; 224
  // workgroups of 32 columns left 32 CUs idle).  Four h row blocks per lane
  // group go out ahead of the weight window; any others follow it.
  if (d.n_experts <= 256)
    MOE_LAUNCH("ffn_decode_down_combine", (ffn_decode_down_combine_kernel<1, 4, 4, 1, 8>),
               dim3((unsigned)(d.hidden / 16)), dim3(512), 0, stream, a);
  else
    MOE_LAUNCH("ffn_decode_down_combine", (ffn_decode_down_combine_kernel<1, 4, 4, kDcMaxExperts / 256, 8>),
               dim3((unsigned)(d.hidden / 16)), dim3(512), 0, stream, a);
  return check_launch("ffn_decode_down_combine");
}

// One token (T = 1, k <= 16): as run_ffn_decode_down_combine with h row j
// belonging to slot j (run_ffn_decode_gateup_one_token's rows) and the
// experts taken from topk_ids.
moe_status_t run_ffn_decode_down_combine_one_token(const moe_dims_t& d, const float* h, const int32_t* topk_ids,
                                                   const uint8_t* w_down, const float* s_down, const float* topk_w,
                                                   uint16_t* out, hipStream_t stream) {
  if (!decode_down_combine_fits(d, 1))
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "decode down+combine: k=%d (max %d), I=%d (max %d)", d.topk, kDcMaxRows,
                d.inter, kDcMaxK);
  DownCombineArgs a{};
  a.h = h; a.ids = topk_ids; a.E = d.n_experts;
  a.w = w_down; a.s = s_down; a.N = d.hidden; a.K = d.inter;
  a.topk_w = topk_w; a.topk = d.topk; a.tokens = 1; a.out = out;
  MOE_LAUNCH("ffn_decode_down_combine", (ffn_decode_down_combine_kernel<1, 4, 4, 1, 8, true>),
             dim3((unsigned)(d.hidden / 16)), dim3(512), 0, stream, a);
  return check_launch("ffn_decode_down_combine");
}

}  // namespace moe
