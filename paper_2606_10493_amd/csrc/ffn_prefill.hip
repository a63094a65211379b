// Prefill-regime expert FFN: block-scaled FP8 MFMA grouped GEMM over the
// expert-sorted rows (the GPU FP8 GEMM path of the paper's FP8 Block Scaling
// Format: FP8 weights and scales from device memory, activations quantized
// to FP8, FP8 x FP8 products with FP32 accumulation; gate and up fused with
// SiLU(gate)*up as in the paper's stage one, down after it).
//
// Tile: 128 expert rows x 256 output columns x one 128-K scale block per
// step, 512 threads (8 waves as 2 x 4).  Both operands are staged through LDS
// (double buffered, one barrier per K step).  Each wave owns 64 rows x 4
// column sub-tiles of 16; every K step issues 16 MFMA 16x16x128 (one scale
// block each) and promotes each result into the fp32 accumulators with the
// block's scale product sa[row,b] * sw[nblock,b] (one FMA per output).
//
// GATEUP: the 256 columns are 128 gate rows and the same 128 up rows of the
// weights, so a workgroup holds one full 128-wide block of h: its epilogue
// computes h = SiLU(G) * U, the per-row amax of the block (lanes, then the
// four column waves through LDS), the scale sh = amax / 448 and the e4m3
// codes qh, staged through LDS and written as 16-byte rows.
// DOWN: the 256 columns are 256 rows of W_down; the epilogue writes fp32.
//
// Work items are (expert m-tile, n-tile) pairs; m-tiles of all experts are
// numbered by an exclusive scan of ceil(M_e / 128) (prefill_tiles_kernel).
// Work items are assigned XCD-major: the hardware deals workgroups to the 8
// XCDs round-robin, so with n real items (read from the tile scan; the grid
// is only an upper bound) item = (block % 8) * ceil(n / 8) + block / 8
// keeps the n-tiles of one m-tile (which share the gathered activation
// rows) and the m-tiles of one expert (which share weights) on one XCD's L2
// while every XCD gets an equal share.
#include "common.h"

namespace moe {

namespace {

constexpr int kBM = 128;
constexpr int kBN = 256;
constexpr int kThreads = 512;
constexpr int kLdsRow = kBlock + 16;  // padded LDS row (bytes) to spread banks
constexpr int kStageA = kBM * kLdsRow;
constexpr int kStageB = kBN * kLdsRow;
constexpr int kStage = kStageA + kStageB;
constexpr int kXcd = 8;

struct PrefillArgs {
  const uint8_t* a;           // e4m3 activations [a_rows, K]
  const float* sa;            // [a_rows, K/128]
  const int32_t* sorted_src;  // GATEUP: A row of sorted row p = sorted_src[p] / topk; DOWN: NULL (A row = p)
  int topk;
  int a_rows;
  const int32_t* offsets;     // [E+1]
  const int32_t* mtile_start; // [E+1] exclusive scan of ceil(M_e/128)
  int E;
  const uint8_t* w0;          // GATEUP: W_gate [E, N, K]; DOWN: W_down [E, N, K]
  const float* s0;
  const uint8_t* w1;          // GATEUP: W_up
  const float* s1;
  int N, K;                   // N: output columns of the expert (I for gate/up, H for down)
  int n_tiles;                // GATEUP: N/128; DOWN: N/256
  float* y;                   // DOWN output fp32 [rows, N]
  uint8_t* qh;                // GATEUP output e4m3 [rows, N]
  float* sh;                  // GATEUP output [rows, N/128]
};

__global__ __launch_bounds__(1024) void prefill_tiles_kernel(const int32_t* __restrict__ offsets, int E,
                                                             int32_t* __restrict__ mtile_start) {
  __shared__ int wave_tot[16];
  const int e = threadIdx.x;
  const int c = (e < E) ? (offsets[e + 1] - offsets[e] + kBM - 1) / kBM : 0;
  int total;
  const int excl = block_exclusive_scan(c, wave_tot, &total);
  if (e < E) mtile_start[e] = excl;
  if (e == 0) mtile_start[E] = total;
}

__device__ __forceinline__ uint4 and4(uint4 v, uint32_t m) {
  return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
}

template <bool GATEUP>
__global__ __launch_bounds__(kThreads) void ffn_prefill_kernel(PrefillArgs p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  __shared__ int arow[kBM];
  __shared__ float rowmax[4][kBM];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int r = lane & 15, kq = lane >> 4;

  // XCD-major work item over the real items (the grid is an upper bound):
  // XCD x takes items [x*per, (x+1)*per) in order.
  const int64_t real = (int64_t)p.mtile_start[p.E] * p.n_tiles;
  const int64_t per = (real + kXcd - 1) / kXcd;
  const int64_t slot = blockIdx.x / kXcd;
  if (slot >= per) return;
  const int64_t item = (int64_t)(blockIdx.x % kXcd) * per + slot;
  if (item >= real) return;
  const int64_t mt_global = item / p.n_tiles;
  const int nt = (int)(item % p.n_tiles);
  // Expert owning this m-tile: last e with mtile_start[e] <= mt_global.
  int lo = 0, hi = p.E - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.mtile_start[mid] <= mt_global) lo = mid; else hi = mid - 1;
  }
  const int e = lo;
  const int m0 = p.offsets[e] + (int)(mt_global - p.mtile_start[e]) * kBM;  // first sorted row of the tile
  const int mc = min(kBM, p.offsets[e + 1] - m0);                            // rows in the tile
  const int nb = p.K / kBlock;

  float* sa_lds = reinterpret_cast<float*>(smem + 2 * kStage);  // [kBM][nb]

  for (int i = tid; i < kBM; i += kThreads) {
    int row = -1;
    if (i < mc) {
      const int src = p.sorted_src ? p.sorted_src[m0 + i] / p.topk : m0 + i;
      row = (src >= 0 && src < p.a_rows) ? src : -1;
    }
    arow[i] = row;
  }
  __syncthreads();
  for (int i = tid; i < kBM * nb; i += kThreads) {
    const int m = i / nb, b = i - m * nb;
    sa_lds[i] = arow[m] >= 0 ? p.sa[(int64_t)arow[m] * nb + b] : 0.0f;
  }

  // Global -> LDS copy assignment: A = 1024 16-byte chunks (2 per thread),
  // B = 2048 chunks (4 per thread); chunk c covers row c/8, bytes 16*(c%8).
  // Rows beyond the expert (or with a bad index) load a valid row and are
  // zeroed after the load, which keeps every load a plain global load.
  const uint8_t* a_src[2];
  uint32_t a_mask[2];
  int a_dst[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = tid + i * kThreads;
    const int row = c >> 3, col = (c & 7) * 16;
    const int ar = arow[row];
    a_mask[i] = ar >= 0 ? 0xffffffffu : 0u;
    a_src[i] = p.a + (int64_t)(ar >= 0 ? ar : 0) * p.K + col;
    a_dst[i] = row * kLdsRow + col;
  }
  const uint8_t* b_src[4];
  int b_dst[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + i * kThreads;
    const int row = c >> 3, col = (c & 7) * 16;
    const uint8_t* base;
    if (GATEUP) {
      const int n = nt * 128 + (row & 127);
      base = (row < 128 ? p.w0 : p.w1) + ((int64_t)e * p.N + n) * p.K;
    } else {
      base = p.w0 + ((int64_t)e * p.N + nt * kBN + row) * p.K;
    }
    b_src[i] = base + col;
    b_dst[i] = kStageA + row * kLdsRow + col;
  }

  // Column sub-tiles of this wave: LDS B rows and their weight-scale source.
  int bsub_row[4];
  const float* wscale[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (GATEUP) {
      bsub_row[j] = (j < 2 ? 0 : 128) + wn * 32 + (j & 1) * 16;
      const int64_t srow = ((int64_t)e * (p.N / kBlock) + nt) * nb;
      wscale[j] = (j < 2 ? p.s0 : p.s1) + srow;
    } else {
      bsub_row[j] = wn * 64 + j * 16;
      const int ncol = nt * kBN + wn * 64;
      wscale[j] = p.s0 + ((int64_t)e * (p.N / kBlock) + ncol / kBlock) * nb;
    }
  }

  v4f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  // Staging registers of one K block (global -> registers -> LDS).  Plain
  // scalars, fully unrolled, so they stay in VGPRs.
  uint4 ra0, ra1, rb0, rb1, rb2, rb3;
#define MOE_PF_GLOAD(BLK)                                                                            \
  do {                                                                                               \
    const int off_ = (BLK) * kBlock;                                                                 \
    ra0 = *reinterpret_cast<const uint4*>(a_src[0] + off_);                                          \
    ra1 = *reinterpret_cast<const uint4*>(a_src[1] + off_);                                          \
    rb0 = *reinterpret_cast<const uint4*>(b_src[0] + off_);                                          \
    rb1 = *reinterpret_cast<const uint4*>(b_src[1] + off_);                                          \
    rb2 = *reinterpret_cast<const uint4*>(b_src[2] + off_);                                          \
    rb3 = *reinterpret_cast<const uint4*>(b_src[3] + off_);                                          \
  } while (0)
#define MOE_PF_LSTORE(STAGE)                                                                         \
  do {                                                                                               \
    uint8_t* st_ = smem + (STAGE) * kStage;                                                          \
    *reinterpret_cast<uint4*>(st_ + a_dst[0]) = and4(ra0, a_mask[0]);                                \
    *reinterpret_cast<uint4*>(st_ + a_dst[1]) = and4(ra1, a_mask[1]);                                \
    *reinterpret_cast<uint4*>(st_ + b_dst[0]) = rb0;                                                 \
    *reinterpret_cast<uint4*>(st_ + b_dst[1]) = rb1;                                                 \
    *reinterpret_cast<uint4*>(st_ + b_dst[2]) = rb2;                                                 \
    *reinterpret_cast<uint4*>(st_ + b_dst[3]) = rb3;                                                 \
  } while (0)

  MOE_PF_GLOAD(0);
  MOE_PF_LSTORE(0);
  __syncthreads();

  for (int b = 0; b < nb; ++b) {
    const int stage = b & 1;
    // The next block's global loads go out first; scheduling barriers keep
    // them above the math and keep the LDS store of the next stage below it,
    // so their latency overlaps this block's MFMAs.  The body is one basic
    // block: the last step re-loads its own block and stores it into the
    // stage nobody reads any more.
    MOE_PF_GLOAD(b + 1 < nb ? b + 1 : b);
    __builtin_amdgcn_sched_barrier(0);
    const uint8_t* sA = smem + stage * kStage;
    const uint8_t* sB = sA + kStageA;
    v8i af[4], bf[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = load_v8i(sA + (wm * 64 + i * 16 + r) * kLdsRow + kq * 32);
#pragma unroll
    for (int j = 0; j < 4; ++j) bf[j] = load_v8i(sB + (bsub_row[j] + r) * kLdsRow + kq * 32);
    float sw[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) sw[j] = wscale[j][b];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float sa[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) sa[q] = sa_lds[(wm * 64 + i * 16 + 4 * kq + q) * nb + b];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const v4f part = mfma_f8_16x16x128(af[i], bf[j]);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][j][q] += part[q] * (sa[q] * sw[j]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    MOE_PF_LSTORE(stage ^ 1);
    __syncthreads();
  }
#undef MOE_PF_GLOAD
#undef MOE_PF_LSTORE

  if (!GATEUP) {
    // y[m0 + row, nt*256 + col]; lane holds rows 4*kq+q of each 16x16 sub-tile, column r.
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = wm * 64 + i * 16 + 4 * kq + q;
        if (row < mc) {
          float* dst = p.y + (int64_t)(m0 + row) * p.N + nt * kBN + wn * 64 + r;
#pragma unroll
          for (int j = 0; j < 4; ++j) dst[j * 16] = acc[i][j][q];
        }
      }
    return;
  }

  // GATEUP epilogue: h = SiLU(G) * U; sub-tiles j = 0,1 are gate, 2,3 up.
  float h[4][2][4];
  float pmax[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float mx = 0.0f;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        h[i][j][q] = silu_mul(acc[i][j][q], acc[i][j + 2][q]);
        mx = fmaxf(mx, fabsf(h[i][j][q]));
      }
      // max over the 16 lanes that share these rows (same kq)
#pragma unroll
      for (int m = 8; m >= 1; m >>= 1) mx = fmaxf(mx, __shfl_xor(mx, m, 16));
      pmax[i][q] = mx;
    }
  if (r == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) rowmax[wn][wm * 64 + i * 16 + 4 * kq + q] = pmax[i][q];
  }
  __syncthreads();
  uint8_t* qtile = smem;  // [kBM][kLdsRow], the K-loop buffers are free now
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int row = wm * 64 + i * 16 + 4 * kq + q;
      const float amax = fmaxf(fmaxf(rowmax[0][row], rowmax[1][row]), fmaxf(rowmax[2][row], rowmax[3][row]));
      const float s = amax / kE4M3Max;
#pragma unroll
      for (int j = 0; j < 2; ++j) qtile[row * kLdsRow + wn * 32 + j * 16 + r] = (uint8_t)quantize_e4m3(h[i][j][q], s);
      if (wn == 0 && r == 0 && row < mc) p.sh[(int64_t)(m0 + row) * (p.N / kBlock) + nt] = s;
    }
  __syncthreads();
  // 128 rows x 128 bytes = 1024 16-byte chunks, 2 per thread.
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = tid + i * kThreads;
    const int row = c >> 3, col = (c & 7) * 16;
    if (row < mc)
      *reinterpret_cast<uint4*>(p.qh + (int64_t)(m0 + row) * p.N + nt * kBlock + col) =
          *reinterpret_cast<const uint4*>(qtile + row * kLdsRow + col);
  }
}

template <bool GATEUP>
moe_status_t launch_prefill(const PrefillArgs& a, int64_t max_mtiles, hipStream_t stream) {
  int64_t grid = max_mtiles * a.n_tiles;
  grid = (grid + kXcd - 1) / kXcd * kXcd;
  if (grid > 0x7fffffff) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: grid too large");
  const size_t lds = 2 * (size_t)kStage + sizeof(float) * (size_t)kBM * (a.K / kBlock);
  if (lds > 150 * 1024) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: K=%d needs %zu bytes of LDS", a.K, lds);
  const hipError_t ae = hipFuncSetAttribute(reinterpret_cast<const void*>(&ffn_prefill_kernel<GATEUP>),
                                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (ae != hipSuccess) return fail(MOE_ERR_HIP, "ffn_prefill: LDS attribute: %s", hipGetErrorString(ae));
  MOE_LAUNCH(GATEUP ? "ffn_prefill_gateup" : "ffn_prefill_down", (ffn_prefill_kernel<GATEUP>), dim3((unsigned)grid), dim3(kThreads), lds, stream, a);
  return check_launch(GATEUP ? "ffn_prefill_gateup" : "ffn_prefill_down");
}

}  // namespace

size_t prefill_tile_workspace(const moe_dims_t& d, int32_t T) {
  (void)T;
  return sizeof(int32_t) * (size_t)(d.n_experts + 1);
}

// Gate/up then down over the expert-sorted rows described by offsets[0..E].
// max_mtiles bounds the number of 128-row tiles over all experts (it sizes
// the grid); a_rows is the number of activation rows (tokens).
moe_status_t run_ffn_prefill_view(const moe_dims_t& d, int64_t max_mtiles, int32_t a_rows, const uint8_t* qx,
                                  const float* sx, const int32_t* offsets, const int32_t* sorted_src,
                                  const uint8_t* w_gate, const float* s_gate, const uint8_t* w_up, const float* s_up,
                                  const uint8_t* w_down, const float* s_down, float* y_rows, uint8_t* qh, float* sh,
                                  int32_t* tiles, hipStream_t stream) {
  if (d.hidden % kBN) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "prefill regime needs H %% 256 == 0 (H=%d)", d.hidden);
  MOE_LAUNCH("prefill_tiles", prefill_tiles_kernel, dim3(1), dim3(1024), 0, stream, offsets, d.n_experts, tiles);
  moe_status_t st = check_launch("prefill_tiles");
  if (st != MOE_OK) return st;

  PrefillArgs g{};
  g.a = qx; g.sa = sx; g.sorted_src = sorted_src; g.topk = d.topk; g.a_rows = a_rows;
  g.offsets = offsets; g.mtile_start = tiles; g.E = d.n_experts;
  g.w0 = w_gate; g.s0 = s_gate; g.w1 = w_up; g.s1 = s_up;
  g.N = d.inter; g.K = d.hidden; g.n_tiles = d.inter / kBlock;
  g.qh = qh; g.sh = sh; g.y = nullptr;
  st = launch_prefill<true>(g, max_mtiles, stream);
  if (st != MOE_OK) return st;

  PrefillArgs dn{};
  dn.a = qh; dn.sa = sh; dn.sorted_src = nullptr; dn.topk = d.topk; dn.a_rows = (int)((int64_t)a_rows * d.topk);
  dn.offsets = offsets; dn.mtile_start = tiles; dn.E = d.n_experts;
  dn.w0 = w_down; dn.s0 = s_down; dn.w1 = nullptr; dn.s1 = nullptr;
  dn.N = d.hidden; dn.K = d.inter; dn.n_tiles = d.hidden / kBN;
  dn.y = y_rows; dn.qh = nullptr; dn.sh = nullptr;
  return launch_prefill<false>(dn, max_mtiles, stream);
}

moe_status_t run_ffn_prefill(const moe_dims_t& d, int32_t T, const uint8_t* qx, const float* sx,
                             const int32_t* offsets, const int32_t* sorted_src, const uint8_t* w_gate,
                             const float* s_gate, const uint8_t* w_up, const float* s_up, const uint8_t* w_down,
                             const float* s_down, float* y_rows, uint8_t* qh, float* sh, int32_t* tiles,
                             hipStream_t stream) {
  const int64_t R = (int64_t)T * d.topk;
  const int64_t max_mtiles = (R + kBM - 1) / kBM + (R < d.n_experts ? R : d.n_experts);
  return run_ffn_prefill_view(d, max_mtiles, T, qx, sx, offsets, sorted_src, w_gate, s_gate, w_up, s_up, w_down,
                              s_down, y_rows, qh, sh, tiles, stream);
}

}  // namespace moe
