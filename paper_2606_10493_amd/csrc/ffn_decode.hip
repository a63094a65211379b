// Decode-regime expert FFN: weight-streaming FP8 MFMA "GEMV" (few tokens per
// expert, HBM bound).
//
// The paper's CPU GEMV keeps three loop levels: output tiles that never cross
// a scale block, K walked in 128-element scale blocks with the block's scale
// applied once to the accumulated partial, and unrolled SIMD dot products
// inside a block (AVX-512 FP8 GEMV Kernel, Tiling and Scale-Block
// Optimizations).  On gfx950 the inner level is one FP8 MFMA 16x16x128: it
// consumes exactly one scale block of 16 weight rows against up to 16 token
// rows, so the fp32 scale product sx[t,b] * sw[n/128,b] is applied once per
// MFMA result, in fp32, as the paper's post-scaling does.
//
// Work item = (active expert, tile of 16*NT weight rows).  A 256-thread
// workgroup (4 waves) splits K and sums the partial accumulators through
// LDS in wave order (deterministic).  Gate/up waves stream contiguous K
// ranges (for the long K of gate/up, strided blocks cost ~3%); down waves
// (short K) take blocks wave, wave + 4, ...  With one 16-token operand
// (MT = 1) the gate/up waves each stream one matrix (waves 0, 1: the K
// halves of W_gate; 2, 3: those of W_up): one sequential stream per wave is
// ~3% faster than two.  With more token operands every wave takes both
// matrices over a K quarter, so the activation fragments are loaded once
// per K block.  Every weight byte is read once; the weights are packed in
// operand tiles (moe_pack_weight), so a wave reads one 16-row x 128-K
// operand as two contiguous 1 KB loads.
//
// Latency is what limits a small GEMV, so the prologue before the first
// weight load is short: every wave finds its expert with ballots over the
// expert offsets (no LDS, no barrier), loads its token indices and then
// issues a window of D K-blocks of weight fragments, gathered activation
// fragments, weight scales and activation scales, all vector loads in one
// in-order stream, so waiting for block j never waits for a later load.
//
// W8A16 (A16): the paper's own GEMV numerics (AVX-512 FP8 GEMV Kernel,
// post-scaling): bf16 activations, the FP8 weights expanded to bf16
// (v_cvt_scalef32_pk_bf16_fp8, exact), bf16 x bf16 products accumulated in
// fp32 over a 128-K block (four MFMA 16x16x32 bf16; the lane's 32 weight
// bytes are split into four 8-element sub-steps and the activations are
// read at the same K positions), and the block's weight scale applied once
// to the block sum.  h is written in bf16 and is the down projection's
// activation.
//
// X1 (one token, no layer prologue): the gate/up kernel quantizes the bf16
// token row into LDS itself (the rule of moe_quant_act, once per workgroup,
// after its first weight block is issued) and takes slot j's expert straight
// from topk_ids: the k slots of one token are distinct experts, so no sort is
// needed, and row j of h is slot j.  Workgroup 0 reports bad ids as the sort
// would; a slot with a bad id gets no row.
//
// GATEUP: the tile holds the same 16*NT rows of W_gate and W_up, and the
// epilogue writes h = SiLU(G) * U in fp32 (bf16 with A16).  Down: h is quantized per row per
// 128 (QH: in this kernel's prologue, for at most kQhRows rows per expert;
// else by a separate launch) and the epilogue writes the fp32 expert rows.
#include "common.h"

namespace moe {

struct DecodeArgs {
  const uint8_t* a;           // e4m3 [a_rows, K]
  const uint16_t* a16;        // A16: bf16 activations [a_rows, K] (a, sa unused)
  const float* sa;            // fp32 [a_rows, K/128]
  const int32_t* sorted_src;  // row p of the expert-sorted order reads A row sorted_src[p]/topk; NULL: A row p
  int topk;
  int a_rows;
  const int32_t* offsets;     // [E+1]
  int E;
  const uint8_t* w0;          // e4m3 [E, N, K], packed tiles
  const float* s0;            // fp32 [E, N/128, K/128]
  const uint8_t* w1;          // second matrix (up) when GATEUP
  const float* s1;
  int N, K;
  float* out;                 // fp32 [rows, N]
  uint16_t* out16;            // A16 GATEUP: bf16 h [rows, N] (out unused)
  const float* hf;            // QH: fp32 h rows [rows, K] quantized in the prologue
  int m_lo, m_hi;             // the launch covers the experts with m_lo <= rows <= m_hi
  const uint16_t* x16;        // X1: bf16 activations of the one token [K], quantized in the kernel
  const int32_t* ids;         // X1: the token's topk expert ids; row j of out is slot j
  int32_t* dev_status;        // X1: MOE_DEV_* bits OR-ed in for bad ids (workgroup 0), or NULL
};

namespace {

constexpr int kWaves = 4;
constexpr int kQhRows = 4;    // QH: rows of h quantized in the down kernel's prologue
constexpr int kQhMaxK = 2048; // QH: 16 lane groups x 128 columns
constexpr int kX1MaxK = 8192; // X1: the token row in LDS, 4 passes of 16 lane groups x 128 columns
constexpr int kX1Passes = kX1MaxK / kBlock / (256 / 16);

// The a-th expert whose row count lies in [m_lo, m_hi] (or -1), the number
// of such experts and the expert's row range, found by one wave with ballots.  The offsets of 256
// experts are loaded in one round trip (4 per lane + the end value), so the
// lookup costs one L2 latency before the weight stream can start.
struct ExpertRef {
  int e, n_active, p0, m;
};

__device__ __forceinline__ ExpertRef find_expert(const int32_t* __restrict__ offsets, int E, int64_t a, int m_lo,
                                                 int m_hi) {
  const int lane = threadIdx.x & 63;
  ExpertRef ref{-1, 0, 0, 0};
  for (int c0 = 0; c0 < E; c0 += 256) {
    int o[5];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int x = c0 + 64 * c + lane;
      o[c] = x <= E ? offsets[x] : 0;
    }
    o[4] = offsets[min(c0 + 256, E)];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int x = c0 + 64 * c + lane;
      const int nxt_first = c < 3 ? __shfl(o[c + 1], 0) : o[4];
      const int up = __shfl_down(o[c], 1);
      const int nxt = lane < 63 ? up : nxt_first;
      const bool on = x < E && nxt - o[c] >= m_lo && nxt - o[c] <= m_hi;
      const unsigned long long bal = __ballot(on);
      const int cnt = __popcll(bal);
      if (ref.e < 0 && a < ref.n_active + cnt) {
        unsigned long long msk = bal;
        for (int i = 0; i < (int)(a - ref.n_active); ++i) msk &= msk - 1ull;
        const int bit = __ffsll((long long)msk) - 1;
        ref.e = c0 + 64 * c + bit;
        ref.p0 = __shfl(o[c], bit);
        ref.m = __shfl(nxt, bit) - ref.p0;
      }
      ref.n_active += cnt;
    }
  }
  return ref;
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Eight e4m3 weight bytes (two dwords) -> eight bf16 values, byte order kept.
__device__ __forceinline__ bf16x8 e4m3x8_to_bf16(int d0, int d1) {
  const bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((unsigned)d0, 1.0f, false);
  const bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((unsigned)d0, 1.0f, true);
  const bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((unsigned)d1, 1.0f, false);
  const bf16x2 e = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((unsigned)d1, 1.0f, true);
  return bf16x8{a[0], a[1], b[0], b[1], c[0], c[1], e[0], e[1]};
}

template <int MT, int NT, bool GATEUP, bool QH, int U, bool A16 = false, bool X1 = false>
__global__ __launch_bounds__(256) void ffn_decode_kernel(DecodeArgs p) {
  static_assert(!QH || (!GATEUP && MT == 1), "QH is the down projection with at most 16 rows");
  static_assert(!(A16 && QH), "W8A16 reads bf16 h rows directly");
  static_assert(!X1 || (GATEUP && MT == 1 && !A16), "X1 is the one-token gate/up");
  static_assert(!GATEUP || NT == 1, "a GATEUP tile is 16 rows of W_gate and of W_up");
  constexpr bool kSplit = GATEUP && MT == 1;  // one matrix per wave (waves 0, 1 gate; 2, 3 up)
  constexpr int G = (GATEUP && !kSplit) ? 2 : 1;  // weight matrices per wave
  constexpr int kPer = G * MT * NT * 4;           // partial results per lane
  __shared__ float red[(kWaves - 1) * kPer * 64];
  __shared__ __attribute__((aligned(16))) uint8_t qh_lds[QH ? kQhRows * kQhMaxK : 16];
  __shared__ float sh_lds[QH ? kQhRows * (kQhMaxK / kBlock) : 1];
  __shared__ __attribute__((aligned(16))) uint8_t qx_lds[X1 ? kX1MaxK : 16];
  __shared__ float sx_lds[X1 ? kX1MaxK / kBlock : 1];

  const int nb = p.K / kBlock;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15;   // row of the A / B fragment this lane loads
  const int kq = lane >> 4;  // K lane group: bytes [16 kq, +16) and [64 + 16 kq, +16) of a block
  const int tiles = p.N / (16 * NT);
  // K blocks of this wave: gate/up (long K) a contiguous half (kSplit) or
  // quarter [kb0, kb0 + nkw); down (short K) blocks wave, wave + 4, ..., so
  // the four waves read neighbouring tiles (measured faster for K = 2048).
  // With kSplit the wave's matrix is W_up for waves 2, 3.
  constexpr bool kContig = GATEUP;
  const int kpart = kSplit ? (wave & 1) : wave, nparts = kSplit ? 2 : kWaves;
  const int kb0 = kContig ? (kpart * nb) / nparts : wave;
  const int kstride = kContig ? 1 : kWaves;
  const int nkw = kContig ? ((kpart + 1) * nb) / nparts - kb0 : (nb - wave + kWaves - 1) / kWaves;
  const bool up_wave = kSplit && (wave >> 1);
  const uint8_t* wfirst_mat = up_wave ? p.w1 : p.w0;
  const float* sfirst_mat = up_wave ? p.s1 : p.s0;

  // X1: the token's bf16 row goes out first, 8 values per lane of each
  // 16-lane group of a 128-column block (blocks past the last load the last
  // again), to be quantized into LDS once the first weights are in flight.
  uint4 xraw[X1 ? kX1Passes : 1];
  if constexpr (X1) {
#pragma unroll
    for (int q = 0; q < kX1Passes; ++q) {
      const int g = min((int)(threadIdx.x >> 4) + q * 16, nb - 1);
      xraw[q] = *reinterpret_cast<const uint4*>(p.x16 + g * kBlock + (threadIdx.x & 15) * 8);
    }
  }
  // X1: item a * tiles + t is slot a's expert (one row, row a of out), with
  // no sort: the slots of one token are distinct experts.  A slot whose id
  // lies outside [0, E) or repeats an earlier slot's has no row (m = 0), as
  // the sort leaves such slots out; workgroup 0 reports them.
  auto slot_ref = [&](int64_t a) {
    const int idv = lane < p.topk ? p.ids[lane] : -1;
    const int e = __shfl(idv, (int)a);
    const bool dup = __ballot(lane < a && idv == e) != 0ull;
    const bool ok = e >= 0 && e < p.E && !dup;
    return ExpertRef{ok ? e : -1, p.topk, (int)a, ok ? 1 : 0};
  };
  if constexpr (X1) {
    if (blockIdx.x == 0 && wave == 0) {
      const int idv = lane < p.topk ? p.ids[lane] : 0;
      uint32_t err = 0;
      bool dup = false;
      for (int i = 0; i < p.topk; ++i) {
        const int o = __shfl(idv, i);
        dup |= i < lane && o == idv;
      }
      if (lane < p.topk) err = (idv < 0 || idv >= p.E) ? MOE_DEV_BAD_EXPERT_ID : dup ? MOE_DEV_DUP_EXPERT_ID : 0u;
      for (int m = 32; m >= 1; m >>= 1) err |= (uint32_t)__shfl_xor((int)err, m, 64);
      if (p.dev_status && err && lane == 0) atomicOr(p.dev_status, (int)err);
    }
  }
  bool x_done = false;  // X1: qx_lds holds the token row

  ExpertRef ref = X1 ? slot_ref(blockIdx.x / tiles) : find_expert(p.offsets, p.E, blockIdx.x / tiles, p.m_lo, p.m_hi);
  const int64_t items = (int64_t)ref.n_active * tiles;

  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    if (item != blockIdx.x) ref = X1 ? slot_ref(item / tiles) : find_expert(p.offsets, p.E, item / tiles, p.m_lo, p.m_hi);
    const int e = ref.e;
    const int n0 = (int)(item % tiles) * 16 * NT;
    const int p0 = ref.p0;
    const int M = ref.m;
    // Lane's byte of the first packed tile of each 16-row operand; the
    // tiles of one 16-row group follow each other along K.
    const uint8_t* wrow0[NT];
    const uint8_t* wrow1[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int64_t grp = ((int64_t)e * p.N + n0 + nt * 16) / 16;
      wrow0[nt] = wfirst_mat + grp * nb * kTileBytes + packed_lane_offset(0, kq, r);
      wrow1[nt] = G == 2 ? p.w1 + grp * nb * kTileBytes + packed_lane_offset(0, kq, r) : nullptr;
    }
    const int64_t srow = ((int64_t)e * (p.N / kBlock) + n0 / kBlock) * nb;

    for (int mb = 0; mb < M; mb += 16 * MT) {
      const int mc = min(M - mb, 16 * MT);
      // Activation rows this lane loads (row r of each sub-tile) and the rows
      // whose outputs it holds (4*kq + i), or -1 beyond the expert's rows.
      // All index loads are issued before any of them is used (clamped
      // indices, no branches), so they cost one round trip together.
      auto load_w = [&](int bk, v8i (&w)[G][NT]) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          w[0][nt] = load_v8i_packed_stream(wrow0[nt] + bk * kTileBytes);
          if (G == 2) w[G - 1][nt] = load_v8i_packed_stream(wrow1[nt] + bk * kTileBytes);
        }
      };
      // The wave's weight scales, lane i holding the scale of its i-th K
      // block (clamped), in one load ahead of the weight stream; the j-th
      // block reads lane j.
      float wsv[G];
      {
        const int sl = min(kb0 + kstride * min(lane, max(nkw - 1, 0)), nb - 1);
        wsv[0] = sfirst_mat[srow + sl];
        if (G == 2) wsv[G - 1] = p.s1[srow + sl];
      }
      auto scales_of = [&](int j, float (&ws)[G]) {
#pragma unroll
        for (int g = 0; g < G; ++g) ws[g] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wsv[g]), j));
      };
      int ta[MT], ts[MT][4];
      int raw[MT][5];
      if (!QH && !X1) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int q = 0; q < 5; ++q) {
            const int m = mt * 16 + (q == 0 ? r : 4 * kq + q - 1);
            const int mm = m < mc ? m : mc - 1;
            raw[mt][q] = p.sorted_src ? p.sorted_src[p0 + mb + mm] : p0 + mb + mm;
          }
      }
      // QH: h values of this lane group (column block qgrp), loaded before the weights.
      const int qsub = threadIdx.x & 15, qgrp = threadIdx.x >> 4;
      const int qcol = qgrp * kBlock + qsub * 8;
      float hv[QH ? kQhRows : 1][8];
      if (QH) {
#pragma unroll
        for (int q = 0; q < kQhRows; ++q) {
          if (q < mc && qcol < p.K) {
            const float* src = p.hf + (int64_t)(p0 + mb + q) * p.K + qcol;
            const float4 x0 = *reinterpret_cast<const float4*>(src);
            const float4 x1 = *reinterpret_cast<const float4*>(src + 4);
            hv[q][0] = x0.x; hv[q][1] = x0.y; hv[q][2] = x0.z; hv[q][3] = x0.w;
            hv[q][4] = x1.x; hv[q][5] = x1.y; hv[q][6] = x1.z; hv[q][7] = x1.w;
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) hv[q][i] = 0.0f;
          }
        }
      }
      // The wave's first weight block goes out now, so the weight stream
      // starts while the index (or h) loads are still in flight.  A wave
      // without K blocks (nb < 4) loads nothing: its block index would lie
      // past the end of the rows.
      v8i wfirst[G][NT];
      if (nkw > 0) load_w(kb0, wfirst);
      __builtin_amdgcn_sched_barrier(0);
      if (X1) {  // the one token row: A row 0, scale row 0
        ta[0] = r == 0 ? 0 : -1;
#pragma unroll
        for (int i = 0; i < 4; ++i) ts[0][i] = (kq == 0 && i == 0) ? 0 : -1;
        if (!x_done) {
          // The token row per 128 -> e4m3 in LDS (the rule of moe_quant_act).
#pragma unroll
          for (int q = 0; q < kX1Passes; ++q) {
            const int g = (int)(threadIdx.x >> 4) + q * 16;
            if (g < nb) {  // whole 16-lane groups
              float v[8];
              bf16x8_to_f32(xraw[q], v);
              uint2 codes;
              const float sc = quant_group8(v, codes);
              *reinterpret_cast<uint2*>(qx_lds + g * kBlock + (threadIdx.x & 15) * 8) = codes;
              if ((threadIdx.x & 15) == 0) sx_lds[g] = sc;
            }
          }
          __syncthreads();
          x_done = true;
        }
      } else if (!QH) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int q = 0; q < 5; ++q) {
            const int m = mt * 16 + (q == 0 ? r : 4 * kq + q - 1);
            const int src = p.sorted_src ? raw[mt][q] / p.topk : raw[mt][q];
            const int v = (m < mc && src >= 0 && src < p.a_rows) ? src : -1;
            if (q == 0) ta[mt] = v; else ts[mt][q - 1] = v;
          }
      }

      if (QH) {
        // h rows of this expert -> e4m3 per 128 in LDS (same rule as moe_quant_rows_f32).
#pragma unroll
        for (int q = 0; q < kQhRows; ++q) {
          if (q < mc && qcol < p.K) {
            float amax = 0.0f;
#pragma unroll
            for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(hv[q][i]));
#pragma unroll
            for (int sh = 8; sh >= 1; sh >>= 1) amax = fmaxf(amax, __shfl_xor(amax, sh, 16));
            const float sc = amax / kE4M3Max;
            const uint32_t lo = quantize4_e4m3(hv[q][0], hv[q][1], hv[q][2], hv[q][3], sc);
            const uint32_t hi = quantize4_e4m3(hv[q][4], hv[q][5], hv[q][6], hv[q][7], sc);
            *reinterpret_cast<uint2*>(qh_lds + q * kQhMaxK + qcol) = make_uint2(lo, hi);
            if (qsub == 0) sh_lds[q * (kQhMaxK / kBlock) + qgrp] = sc;
          }
        }
        __syncthreads();
      }

      v4f acc[G][MT][NT];
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) acc[g][mt][nt] = v4f{0.f, 0.f, 0.f, 0.f};

      // Multiply K block bk (weights in w, ws) into the accumulators.
      auto compute_block = [&](int bk, const v8i (&w)[G][NT], const float (&ws)[G]) {
        v8i afrag[MT];
        float sa[MT][4];
        if (QH) {
          // Rows beyond kQhRows read a valid LDS row; their outputs are never stored.
          const int qr = r < kQhRows ? r : kQhRows - 1;
          afrag[0] = load_v8i_ksplit(qh_lds + qr * kQhMaxK + bk * kBlock + kq * 16);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = 4 * kq + i;
            sa[0][i] = row < kQhRows ? sh_lds[row * (kQhMaxK / kBlock) + bk] : 0.0f;
          }
        } else if (X1) {
          afrag[0] = ta[0] >= 0 ? load_v8i_ksplit(qx_lds + bk * kBlock + kq * 16) : v8i{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
          for (int i = 0; i < 4; ++i) sa[0][i] = ts[0][i] >= 0 ? sx_lds[bk] : 0.0f;
        } else if (!A16) {
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            afrag[mt] = ta[mt] >= 0 ? load_v8i_ksplit(p.a + (int64_t)ta[mt] * p.K + bk * kBlock + kq * 16)
                                    : v8i{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 4; ++i) sa[mt][i] = ts[mt][i] >= 0 ? p.sa[(int64_t)ts[mt][i] * nb + bk] : 0.0f;
          }
        }
        if constexpr (A16) {
          // Activations at the weight bytes' K positions: sub-step s covers
          // weight dwords 2s, 2s+1, i.e. K 16kq + [0,8), 16kq + [8,16),
          // 64 + 16kq + [0,8), 64 + 16kq + [8,16) of the block.
          bf16x8 a16[MT][4];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            if (ta[mt] >= 0) {
              const uint16_t* src = p.a16 + (int64_t)ta[mt] * p.K + bk * kBlock + 16 * kq;
              a16[mt][0] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(src));
              a16[mt][1] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(src + 8));
              a16[mt][2] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(src + 64));
              a16[mt][3] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(src + 72));
            } else {
#pragma unroll
              for (int q = 0; q < 4; ++q) a16[mt][q] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
            }
          }
#pragma unroll
          for (int g = 0; g < G; ++g)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              bf16x8 wb[4];
#pragma unroll
              for (int q = 0; q < 4; ++q) wb[q] = e4m3x8_to_bf16(w[g][nt][2 * q], w[g][nt][2 * q + 1]);
#pragma unroll
              for (int mt = 0; mt < MT; ++mt) {
                v4f part = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < 4; ++q) part = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a16[mt][q], wb[q], part, 0, 0, 0);
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[g][mt][nt][i] += part[i] * ws[g];
              }
            }
        } else {
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
              for (int nt = 0; nt < NT; ++nt) {
                const v4f part = mfma_f8_16x16x128(afrag[mt], w[g][nt]);
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[g][mt][nt][i] += part[i] * (sa[mt][i] * ws[g]);
              }
        }
      };

      // K loop: block 0 was loaded above; each later block's loads are
      // issued at the top of its iteration and the unrolled copies let the
      // compiler hoist the next blocks' loads.
      if (nkw > 0) {
        float ws[G];
        scales_of(0, ws);
        compute_block(kb0, wfirst, ws);
      }
#pragma unroll U
      for (int j = 1; j < nkw; ++j) {
        const int bk = kb0 + kstride * j;
        v8i w[G][NT];
        float ws[G];
        load_w(bk, w);
        scales_of(j, ws);
        compute_block(bk, w, ws);
      }

      // Cross-wave reduction in wave order 0, 1, 2, 3 (kSplit: gate = waves
      // 0 + 1, up = waves 2 + 3).
      if (wave > 0) {
        float* dst = red + (wave - 1) * kPer * 64;
        int q = 0;
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
              for (int i = 0; i < 4; ++i) dst[(q++) * 64 + lane] = acc[g][mt][nt][i];
      }
      __syncthreads();
      if (wave == 0) {
        v4f up[MT][NT];  // kSplit: the up result
        {
          const float* s1 = red + 0 * kPer * 64;
          const float* s2 = red + 1 * kPer * 64;
          const float* s3 = red + 2 * kPer * 64;
          int q = 0;
#pragma unroll
          for (int g = 0; g < G; ++g)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
              for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int i = 0; i < 4; ++i, ++q) {
                  acc[g][mt][nt][i] += s1[q * 64 + lane];
                  if (kSplit) {
                    up[mt][nt][i] = s2[q * 64 + lane] + s3[q * 64 + lane];
                  } else {
                    acc[g][mt][nt][i] += s2[q * 64 + lane];
                    acc[g][mt][nt][i] += s3[q * 64 + lane];
                  }
                }
        }
        // Output layout of the 16x16 MFMA: lane l holds rows 4*(l/16)+i, column l%16.
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int m = mt * 16 + 4 * kq + i;
              if (m < mc) {
                float v;
                if (kSplit) v = silu_mul(acc[0][mt][nt][i], up[mt][nt][i]);
                else if (GATEUP) v = silu_mul(acc[0][mt][nt][i], acc[G - 1][mt][nt][i]);
                else v = acc[0][mt][nt][i];
                const int64_t at = (int64_t)(p0 + mb + m) * p.N + n0 + nt * 16 + r;
                if (A16 && GATEUP) p.out16[at] = f32_to_bf16_rne(v);
                else p.out[at] = v;
              }
            }
      }
      __syncthreads();
    }
  }
}

template <int MT, int NT, bool GATEUP, bool QH, int U, bool A16 = false, bool X1 = false>
moe_status_t launch_decode(const DecodeArgs& a, int64_t max_items, hipStream_t stream) {
  const int64_t grid = max_items < 2048 ? max_items : 2048;
  if (grid <= 0) return MOE_OK;
  const char* name = A16 ? (GATEUP ? "ffn_decode_w8a16_gateup" : "ffn_decode_w8a16_down")
                         : (GATEUP ? "ffn_decode_gateup" : "ffn_decode_down");
  MOE_LAUNCH(name, (ffn_decode_kernel<MT, NT, GATEUP, QH, U, A16, X1>), dim3((unsigned)grid), dim3(256), 0, stream,
             a);
  return check_launch(name);
}

// One operation (gate/up or down) over the active experts, one launch per
// row-count class: experts with up to 16 rows take the one-operand kernel
// (every expert when T <= 16), 17-32 rows two operands, more rows four, so
// that the many experts with few rows of a mixed batch run at the register
// budget (and occupancy) of the one-operand kernel.  Each launch covers
// only its experts; an expert has at most T rows.
template <int NT, bool GATEUP, bool QH, int U1, int U24, bool A16 = false>
moe_status_t launch_by_rows(DecodeArgs a, int32_t T, int64_t R, int tiles_per_expert, hipStream_t stream) {
  auto items = [&](int lo) {  // experts with at least lo rows, at most E
    const int64_t n = R / lo;
    return (n < a.E ? n : (int64_t)a.E) * tiles_per_expert;
  };
  a.m_lo = 1;
  a.m_hi = 16;
  moe_status_t st = launch_decode<1, NT, GATEUP, QH, U1, A16>(a, items(1), stream);
  if (st != MOE_OK || T <= 16) return st;
  a.m_lo = 17;
  a.m_hi = 32;
  st = launch_decode<2, NT, GATEUP, false, U24, A16>(a, items(17), stream);
  if (st != MOE_OK || T <= 32) return st;
  a.m_lo = 33;
  a.m_hi = 0x7fffffff;
  return launch_decode<4, NT, GATEUP, false, U24, A16>(a, items(33), stream);
}

}  // namespace

// Shapes the decode kernels take: a wave's weight scales sit one per lane,
// so at most 64 K blocks per wave (gate/up waves may take K halves).
moe_status_t decode_shape_check(const moe_dims_t& d) {
  if (d.hidden / kBlock > 64 * 2 || d.inter / kBlock > 64 * kWaves)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "decode regime supports H <= %d and I <= %d", 64 * 2 * kBlock,
                64 * kWaves * kBlock);
  return MOE_OK;
}

// Decode-regime gate/up: h = SiLU(G) * U in fp32, one row per expert-sorted slot.
moe_status_t run_ffn_decode_gateup(const moe_dims_t& d, int32_t T, const uint8_t* qx, const float* sx,
                                   const int32_t* offsets, const int32_t* sorted_src, const uint8_t* w_gate,
                                   const float* s_gate, const uint8_t* w_up, const float* s_up, float* h,
                                   hipStream_t stream) {
  const int64_t R = (int64_t)T * d.topk;
  moe_status_t st0 = decode_shape_check(d);
  if (st0 != MOE_OK) return st0;
  DecodeArgs g{};
  g.a = qx; g.sa = sx; g.sorted_src = sorted_src; g.topk = d.topk; g.a_rows = T;
  g.offsets = offsets; g.E = d.n_experts;
  g.w0 = w_gate; g.s0 = s_gate; g.w1 = w_up; g.s1 = s_up;
  g.N = d.inter; g.K = d.hidden; g.out = h;
  return launch_by_rows<1, true, false, 3, 2>(g, T, R, d.inter / 16, stream);
}

// One token without the layer prologue: the gate/up GEMV quantizes the bf16
// row and takes slot j's expert from topk_ids itself (no sort: one token's
// slots are distinct experts); h row j belongs to slot j, and a slot with a
// bad id has no row.  Needs K = H <= kX1MaxK; callers check
// decode_one_token_fits.
bool decode_one_token_fits(const moe_dims_t& d) { return d.hidden <= kX1MaxK; }

moe_status_t run_ffn_decode_gateup_one_token(const moe_dims_t& d, const uint16_t* x, const int32_t* topk_ids,
                                             int32_t* dev_status, const uint8_t* w_gate, const float* s_gate,
                                             const uint8_t* w_up, const float* s_up, float* h, hipStream_t stream) {
  moe_status_t st0 = decode_shape_check(d);
  if (st0 != MOE_OK) return st0;
  if (!decode_one_token_fits(d))
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "one-token decode: H=%d > %d", d.hidden, kX1MaxK);
  DecodeArgs g{};
  g.x16 = x; g.ids = topk_ids; g.dev_status = dev_status; g.topk = d.topk; g.a_rows = 1; g.E = d.n_experts;
  g.w0 = w_gate; g.s0 = s_gate; g.w1 = w_up; g.s1 = s_up;
  g.N = d.inter; g.K = d.hidden; g.out = h;
  return launch_decode<1, 1, true, false, 3, false, true>(g, (int64_t)d.topk * (d.inter / 16), stream);
}

// Decode-regime FFN: gate/up -> h (fp32) -> quantize h -> down.
moe_status_t run_ffn_decode(const moe_dims_t& d, int32_t T, const uint8_t* qx, const float* sx,
                            const int32_t* offsets, const int32_t* sorted_src, const uint8_t* w_gate,
                            const float* s_gate, const uint8_t* w_up, const float* s_up, const uint8_t* w_down,
                            const float* s_down, float* y_rows, float* h, uint8_t* qh, float* sh,
                            hipStream_t stream) {
  const int64_t R = (int64_t)T * d.topk;
  const int64_t max_active = R < d.n_experts ? R : d.n_experts;
  moe_status_t st = run_ffn_decode_gateup(d, T, qx, sx, offsets, sorted_src, w_gate, s_gate, w_up, s_up, h, stream);
  if (st != MOE_OK) return st;

  DecodeArgs dn{};
  dn.a = qh; dn.sa = sh; dn.sorted_src = nullptr; dn.topk = d.topk; dn.a_rows = (int)R;
  dn.offsets = offsets; dn.E = d.n_experts;
  dn.w0 = w_down; dn.s0 = s_down; dn.w1 = nullptr; dn.s1 = nullptr;
  dn.N = d.hidden; dn.K = d.inter; dn.out = y_rows; dn.hf = h;
  const int64_t dn_items = max_active * (d.hidden / 32);
  // Up to kQhRows tokens (so at most kQhRows rows per expert) the down kernel
  // quantizes h itself; above that a separate launch writes qh, sh first.
  if (T <= kQhRows && d.inter <= kQhMaxK) {
    dn.m_lo = 1;
    dn.m_hi = 0x7fffffff;
    return launch_decode<1, 2, false, true, 4>(dn, dn_items, stream);
  }
  st = moe_quant_rows_f32(h, (int32_t)R, d.inter, qh, sh, stream);
  if (st != MOE_OK) return st;
  return launch_by_rows<2, false, false, 4, 2>(dn, T, R, d.hidden / 32, stream);
}

// W8A16 decode FFN: bf16 activations, gate/up -> h (bf16) -> down.
moe_status_t run_ffn_decode_w8a16(const moe_dims_t& d, int32_t T, const uint16_t* x, const int32_t* offsets,
                                  const int32_t* sorted_src, const uint8_t* w_gate, const float* s_gate,
                                  const uint8_t* w_up, const float* s_up, const uint8_t* w_down,
                                  const float* s_down, float* y_rows, uint16_t* h16, hipStream_t stream) {
  const int64_t R = (int64_t)T * d.topk;
  moe_status_t st0 = decode_shape_check(d);
  if (st0 != MOE_OK) return st0;
  DecodeArgs g{};
  g.a16 = x; g.sorted_src = sorted_src; g.topk = d.topk; g.a_rows = T;
  g.offsets = offsets; g.E = d.n_experts;
  g.w0 = w_gate; g.s0 = s_gate; g.w1 = w_up; g.s1 = s_up;
  g.N = d.inter; g.K = d.hidden; g.out16 = h16;
  moe_status_t st = launch_by_rows<1, true, false, 3, 2, true>(g, T, R, d.inter / 16, stream);
  if (st != MOE_OK) return st;
  DecodeArgs dn{};
  dn.a16 = h16; dn.sorted_src = nullptr; dn.topk = d.topk; dn.a_rows = (int)R;
  dn.offsets = offsets; dn.E = d.n_experts;
  dn.w0 = w_down; dn.s0 = s_down;
  dn.N = d.hidden; dn.K = d.inter; dn.out = y_rows;
  return launch_by_rows<2, false, false, 4, 2, true>(dn, T, R, d.hidden / 32, stream);
}

}  // namespace moe
