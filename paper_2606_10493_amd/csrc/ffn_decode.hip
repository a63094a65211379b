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
// workgroup (4 waves) splits K: wave w takes blocks b = w, w+4, ...; the
// partial accumulators are summed through LDS in wave order (deterministic).
// Every weight byte is read once, with each lane loading 32 contiguous bytes
// of one row (16 rows x 128 bytes = 16 full cache lines per wave-load).
// Token rows (at most 16*MT per pass) are gathered from the quantized
// activations; rows beyond the expert's count are zero.
//
// GATEUP: the tile holds the same 16*NT rows of W_gate and W_up, and the
// epilogue writes h = SiLU(G) * U in fp32 (quantized per 128 by the next
// launch).  Down: the epilogue writes the fp32 expert rows.
#include "common.h"

namespace moe {

struct DecodeArgs {
  const uint8_t* a;           // e4m3 [a_rows, K]
  const float* sa;            // fp32 [a_rows, K/128]
  const int32_t* sorted_src;  // row p of the expert-sorted order reads A row sorted_src[p]/topk; NULL: A row p
  int topk;
  int a_rows;
  const int32_t* offsets;     // [E+1]
  int E;
  const uint8_t* w0;          // e4m3 [E, N, K]
  const float* s0;            // fp32 [E, N/128, K/128]
  const uint8_t* w1;          // second matrix (up) when GATEUP
  const float* s1;
  int N, K;
  float* out;                 // fp32 [rows, N]
};

namespace {

constexpr int kWaves = 4;
constexpr int kMaxExperts = 1024;

// Active experts (non-empty rows) in ascending id order, compacted in LDS.
__device__ int list_active_experts(const int32_t* __restrict__ offsets, int E, int* active, int* wave_tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int base = 0;
  for (int e0 = 0; e0 < E; e0 += 256) {
    const int e = e0 + threadIdx.x;
    const bool on = (e < E) && (offsets[e + 1] > offsets[e]);
    const unsigned long long bal = __ballot(on);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wave_tot[wave] = __popcll(bal);
    __syncthreads();
    int off = base;
    for (int w = 0; w < wave; ++w) off += wave_tot[w];
    if (on) active[off + before] = e;
    base += wave_tot[0] + wave_tot[1] + wave_tot[2] + wave_tot[3];
    __syncthreads();
  }
  return base;
}

template <int MT, int NT, bool GATEUP>
__global__ __launch_bounds__(256) void ffn_decode_kernel(DecodeArgs p) {
  constexpr int G = GATEUP ? 2 : 1;
  constexpr int kRows = 16 * MT;
  extern __shared__ float smem[];
  __shared__ int active[kMaxExperts];
  __shared__ int wave_tot[kWaves];
  __shared__ int tok[kRows];

  const int nb = p.K / kBlock;
  float* sa_lds = smem;                        // [kRows][nb]
  float* red = smem + kRows * nb;              // [kWaves-1][G][MT][NT][4][64]

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane & 15;   // row of the A / B fragment this lane loads
  const int kq = lane >> 4;  // 32-byte K slice of the block this lane loads

  const int n_active = list_active_experts(p.offsets, p.E, active, wave_tot);
  const int tiles = p.N / (16 * NT);
  const int64_t items = (int64_t)n_active * tiles;

  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int e = active[item / tiles];
    const int n0 = (int)(item % tiles) * 16 * NT;
    const int p0 = p.offsets[e];
    const int M = p.offsets[e + 1] - p0;
    const uint8_t* wrow0[NT];
    const uint8_t* wrow1[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int64_t row = (int64_t)e * p.N + n0 + nt * 16 + r;
      wrow0[nt] = p.w0 + row * p.K + kq * 32;
      wrow1[nt] = GATEUP ? p.w1 + row * p.K + kq * 32 : nullptr;
    }
    const int64_t srow = ((int64_t)e * (p.N / kBlock) + n0 / kBlock) * nb;
    const float* sw0 = p.s0 + srow;
    const float* sw1 = GATEUP ? p.s1 + srow : nullptr;

    for (int mb = 0; mb < M; mb += kRows) {
      const int mc = min(M - mb, kRows);
      for (int i = threadIdx.x; i < kRows; i += 256) {
        int arow = -1;
        if (i < mc) {
          const int src = p.sorted_src ? p.sorted_src[p0 + mb + i] / p.topk : p0 + mb + i;
          arow = (src >= 0 && src < p.a_rows) ? src : -1;
        }
        tok[i] = arow;
      }
      __syncthreads();
      for (int i = threadIdx.x; i < kRows * nb; i += 256) {
        const int m = i / nb, b = i - m * nb;
        sa_lds[i] = tok[m] >= 0 ? p.sa[(int64_t)tok[m] * nb + b] : 0.0f;
      }
      const uint8_t* arow_ptr[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int t = tok[mt * 16 + r];
        arow_ptr[mt] = t >= 0 ? p.a + (int64_t)t * p.K + kq * 32 : nullptr;
      }
      __syncthreads();

      v4f acc[G][MT][NT];
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) acc[g][mt][nt] = v4f{0.f, 0.f, 0.f, 0.f};

      v8i bcur[G][NT], bnext[G][NT];
      int b = wave;
      if (b < nb) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          bcur[0][nt] = load_v8i(wrow0[nt] + b * kBlock);
          if (GATEUP) bcur[G - 1][nt] = load_v8i(wrow1[nt] + b * kBlock);
        }
      }
      for (; b < nb; b += kWaves) {
        const int bn = b + kWaves;
        if (bn < nb) {
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            bnext[0][nt] = load_v8i(wrow0[nt] + bn * kBlock);
            if (GATEUP) bnext[G - 1][nt] = load_v8i(wrow1[nt] + bn * kBlock);
          }
        }
        v8i afrag[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          if (arow_ptr[mt]) {
            afrag[mt] = load_v8i(arow_ptr[mt] + b * kBlock);
          } else {
            afrag[mt] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
          }
        }
        float ws[G];
        ws[0] = sw0[b];
        if (GATEUP) ws[G - 1] = sw1[b];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          float sa[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) sa[i] = sa_lds[(mt * 16 + 4 * kq + i) * nb + b];
#pragma unroll
          for (int g = 0; g < G; ++g)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              const v4f part = mfma_f8_16x16x128(afrag[mt], bcur[g][nt]);
#pragma unroll
              for (int i = 0; i < 4; ++i) acc[g][mt][nt][i] += part[i] * (sa[i] * ws[g]);
            }
        }
        if (bn < nb) {
#pragma unroll
          for (int g = 0; g < G; ++g)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) bcur[g][nt] = bnext[g][nt];
        }
      }

      // Cross-wave reduction in wave order 0, 1, 2, 3.
      constexpr int kPer = G * MT * NT * 4;
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
#pragma unroll
        for (int w = 0; w < kWaves - 1; ++w) {
          const float* src = red + w * kPer * 64;
          int q = 0;
#pragma unroll
          for (int g = 0; g < G; ++g)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
              for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[g][mt][nt][i] += src[(q++) * 64 + lane];
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
                const float v = GATEUP ? silu_mul(acc[0][mt][nt][i], acc[G - 1][mt][nt][i]) : acc[0][mt][nt][i];
                p.out[(int64_t)(p0 + mb + m) * p.N + n0 + nt * 16 + r] = v;
              }
            }
      }
      __syncthreads();
    }
  }
}

template <int MT, int NT, bool GATEUP>
moe_status_t launch_decode(const DecodeArgs& a, int64_t max_items, hipStream_t stream) {
  constexpr int G = GATEUP ? 2 : 1;
  const int nb = a.K / kBlock;
  const size_t lds = sizeof(float) * ((size_t)16 * MT * nb + (size_t)(kWaves - 1) * G * MT * NT * 4 * 64);
  const int64_t grid = max_items < 2048 ? max_items : 2048;
  if (grid <= 0) return MOE_OK;
  hipLaunchKernelGGL((ffn_decode_kernel<MT, NT, GATEUP>), dim3((unsigned)grid), dim3(256), lds, stream, a);
  return check_launch(GATEUP ? "ffn_decode_gateup" : "ffn_decode_down");
}

}  // namespace

// Decode-regime FFN: gate/up -> h (fp32) -> quantize h -> down.
moe_status_t run_ffn_decode(const moe_dims_t& d, int32_t T, const uint8_t* qx, const float* sx,
                            const int32_t* offsets, const int32_t* sorted_src, const uint8_t* w_gate,
                            const float* s_gate, const uint8_t* w_up, const float* s_up, const uint8_t* w_down,
                            const float* s_down, float* y_rows, float* h, uint8_t* qh, float* sh,
                            hipStream_t stream) {
  const int64_t R = (int64_t)T * d.topk;
  const int64_t max_active = R < d.n_experts ? R : d.n_experts;
  DecodeArgs g{};
  g.a = qx; g.sa = sx; g.sorted_src = sorted_src; g.topk = d.topk; g.a_rows = T;
  g.offsets = offsets; g.E = d.n_experts;
  g.w0 = w_gate; g.s0 = s_gate; g.w1 = w_up; g.s1 = s_up;
  g.N = d.inter; g.K = d.hidden; g.out = h;
  moe_status_t st;
  const int64_t gu_items = max_active * (d.inter / 16);
  if (T <= 16) st = launch_decode<1, 1, true>(g, gu_items, stream);
  else if (T <= 32) st = launch_decode<2, 1, true>(g, gu_items, stream);
  else st = launch_decode<4, 1, true>(g, gu_items, stream);
  if (st != MOE_OK) return st;

  st = moe_quant_rows_f32(h, (int32_t)R, d.inter, qh, sh, stream);
  if (st != MOE_OK) return st;

  DecodeArgs dn{};
  dn.a = qh; dn.sa = sh; dn.sorted_src = nullptr; dn.topk = d.topk; dn.a_rows = (int)R;
  dn.offsets = offsets; dn.E = d.n_experts;
  dn.w0 = w_down; dn.s0 = s_down; dn.w1 = nullptr; dn.s1 = nullptr;
  dn.N = d.hidden; dn.K = d.inter; dn.out = y_rows;
  const int64_t dn_items = max_active * (d.hidden / 32);
  if (T <= 16) return launch_decode<1, 2, false>(dn, dn_items, stream);
  if (T <= 32) return launch_decode<2, 2, false>(dn, dn_items, stream);
  return launch_decode<4, 2, false>(dn, dn_items, stream);
}

}  // namespace moe
