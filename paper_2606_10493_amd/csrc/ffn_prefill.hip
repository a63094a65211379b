// Prefill-regime expert FFN: block-scaled FP8 MFMA grouped GEMM over the
// expert-sorted rows (the GPU FP8 GEMM path of the paper's FP8 Block Scaling
// Format: FP8 weights and scales from device memory, activations quantized
// to FP8, FP8 x FP8 products with FP32 accumulation; gate and up fused with
// SiLU(gate)*up as in the paper's stage one, down after it).
//
// The products are formed transposed, D = W x X^T: the MFMA's A operand is
// 16 weight rows (output channels), its B operand 16 expert rows (tokens).
// A lane's four results then share one token and lie inside one 128-channel
// weight-scale block, so the per-block scale of a result is (the lane's
// token scale) x (a wave-uniform weight scale).
//
// Tile: 256 weight rows x 128 expert rows x one 128-K scale block per step,
// 512 threads (8 waves).  Wave w owns 32 weight rows (two 16-row MFMA
// operands) against all 128 expert rows (eight 16-row operands): 16 MFMA
// 16x16x128 per K step, each promoted into fp32 accumulators with one FMA
// per result.  The weights are packed in operand tiles (moe_pack_weight),
// so they go from global memory straight into the MFMA operand registers
// with two contiguous 1 KB wave loads per operand (no wave shares them),
// through a ring of kRing K blocks loaded kRing - 1 steps ahead.  Only the
// expert rows, which all waves read, are staged through LDS (double
// buffered, one barrier per K step; loaded as whole 128-byte row pieces),
// and their scales sit in LDS transposed, [K block][row].
//
// GATEUP: wave w's rows are gate rows nt*128 + 16w + [0, 16) and the same up
// rows, so a workgroup holds one full 128-wide block of h: its epilogue
// computes h = SiLU(G) * U, the per-row amax of the block (lanes, then the
// eight waves through LDS), the scale sh = amax / 448 and the e4m3 codes qh,
// staged through LDS and written as 16-byte rows.
// DOWN: wave w's rows are W_down rows nt*256 + 32w + [0, 32); the epilogue
// writes fp32 in 16-byte pieces.
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

constexpr int kBM = 128;                // expert rows (tokens) per tile
constexpr int kBN = 256;                // weight rows per tile
constexpr int kThreads = 512;           // 8 waves x 32 weight rows
constexpr int kLdsRow = kBlock + 16;    // padded LDS row (bytes) to spread banks
constexpr int kStage = kBM * kLdsRow;   // one K block of the expert rows
constexpr int kSaStride = kBM + 1;      // floats per K block of the row-scale table
constexpr int kRing = 4;                // weight K blocks in registers
constexpr int kXcd = 8;
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct PrefillArgs {
  const uint8_t* a;           // e4m3 activations [a_rows, K]
  const float* sa;            // [a_rows, K/128]
  const int32_t* sorted_src;  // GATEUP: A row of sorted row p = sorted_src[p] / topk; DOWN: NULL (A row = p)
  int topk;
  int a_rows;
  const int32_t* offsets;     // [E+1]
  const int32_t* mtile_start; // [E+1] exclusive scan of ceil(M_e/128)
  int E;
  const uint8_t* w0;          // GATEUP: W_gate [E, N, K]; DOWN: W_down [E, N, K]; packed tiles
  const float* s0;
  const uint8_t* w1;          // GATEUP: W_up, packed tiles
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

// Raw buffer view of [base, base + bytes): loads outside it return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_view(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, kRsrcWord3);
}

// One MFMA operand of K block b from a packed weight tile: voff addresses
// byte 16*lane of the operand's first tile, the tiles of one 16-row group
// follow each other along K.
__device__ __forceinline__ v8i load_operand(__amdgpu_buffer_rsrc_t r, uint32_t voff, int b) {
  const u32x4 lo = __builtin_amdgcn_raw_buffer_load_b128(r, voff, b * kTileBytes, 0);
  const u32x4 hi = __builtin_amdgcn_raw_buffer_load_b128(r, voff + 1024, b * kTileBytes, 0);
  v8i o;
  o[0] = lo[0]; o[1] = lo[1]; o[2] = lo[2]; o[3] = lo[3];
  o[4] = hi[0]; o[5] = hi[1]; o[6] = hi[2]; o[7] = hi[3];
  return o;
}

template <bool GATEUP>
__global__ __launch_bounds__(kThreads) void ffn_prefill_kernel(PrefillArgs p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  __shared__ int arow[kBM];
  __shared__ float rowmax[8][kBM];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
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

  float* sa_lds = reinterpret_cast<float*>(smem + 2 * kStage);  // [nb][kSaStride]
  float* sw_lds = sa_lds + nb * kSaStride;                       // [2][nb]

  for (int i = tid; i < kBM; i += kThreads) {
    int row = -1;
    if (i < mc) {
      const int src = p.sorted_src ? p.sorted_src[m0 + i] / p.topk : m0 + i;
      row = (src >= 0 && src < p.a_rows) ? src : -1;
    }
    arow[i] = row;
  }
  // Weight scales of the tile's two 128-row blocks: GATEUP gate and up block
  // nt; DOWN blocks 2nt and 2nt + 1 (waves 0-3 and 4-7).
  for (int i = tid; i < 2 * nb; i += kThreads) {
    const int h = i / nb, b = i - h * nb;
    const int64_t wrow = (int64_t)e * (p.N / kBlock) + (GATEUP ? nt : 2 * nt + h);
    sw_lds[i] = ((GATEUP && h) ? p.s1 : p.s0)[wrow * nb + b];
  }
  __syncthreads();
  for (int i = tid; i < kBM * nb; i += kThreads) {
    const int m = i / nb, b = i - m * nb;
    sa_lds[b * kSaStride + m] = arow[m] >= 0 ? p.sa[(int64_t)arow[m] * nb + b] : 0.0f;
  }

  // Expert rows: 1024 16-byte chunks per K block, 2 per thread; chunk c
  // covers row c/8, bytes 16*(c%8).  Rows beyond the expert (or with a bad
  // index) load row 0 instead: their codes are finite and their scale in
  // sa_lds is 0, so their products promote to exactly 0, and only rows
  // below mc are written.
  const uint8_t* a_src[2];
  int a_dst[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = tid + i * kThreads;
    const int row = c >> 3, col = (c & 7) * 16;
    const int ar = arow[row];
    a_src[i] = p.a + (int64_t)(ar >= 0 ? ar : 0) * p.K + col;
    a_dst[i] = row * kLdsRow + col;
  }

  // This wave's two 16-row weight operands (f = 0, 1), as buffer views of
  // one expert's packed matrix, and the LDS row of their weight scales.
  const uint32_t wbytes = (uint32_t)p.N * (uint32_t)p.K;
  __amdgpu_buffer_rsrc_t wv[2];
  uint32_t w_off[2];
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    // 16-row group of the operand: GATEUP rows nt*128 + 16w, DOWN rows nt*256 + 32w + 16f.
    const int g = GATEUP ? nt * (kBlock / 16) + wave : nt * (kBN / 16) + wave * 2 + f;
    wv[f] = buffer_view((GATEUP && f ? p.w1 : p.w0) + (int64_t)e * wbytes, wbytes);
    w_off[f] = (uint32_t)g * (uint32_t)nb * kTileBytes + lane * 16;
  }
  const float* swf0 = sw_lds + (GATEUP ? 0 : (wave >> 2)) * nb;
  const float* swf1 = sw_lds + (GATEUP ? 1 : (wave >> 2)) * nb;

  v4f acc[2][8];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[f][i] = v4f{0.f, 0.f, 0.f, 0.f};

  v8i wr[kRing][2];
  u32x4 ra[kRing][2];  // ext vectors: an array of HIP's uint4 structs would not stay in registers
#define MOE_PF_WLOAD(SLOT, BLK)                        \
  do {                                                 \
    wr[SLOT][0] = load_operand(wv[0], w_off[0], BLK);  \
    wr[SLOT][1] = load_operand(wv[1], w_off[1], BLK);  \
  } while (0)
#define MOE_PF_ALOAD(SLOT, BLK)                                                         \
  do {                                                                                  \
    ra[SLOT][0] = *reinterpret_cast<const u32x4*>(a_src[0] + (int64_t)(BLK) * kBlock);  \
    ra[SLOT][1] = *reinterpret_cast<const u32x4*>(a_src[1] + (int64_t)(BLK) * kBlock);  \
  } while (0)
#define MOE_PF_ASTORE(SLOT, STAGE)                                                         \
  do {                                                                                     \
    uint8_t* st_ = smem + (STAGE) * kStage;                                                \
    *reinterpret_cast<u32x4*>(st_ + a_dst[0]) = ra[SLOT][0];                               \
    *reinterpret_cast<u32x4*>(st_ + a_dst[1]) = ra[SLOT][1];                               \
  } while (0)
  // One K step b using register slot U (= b % kRing).  The loads of block
  // b + kRing - 1 (expert rows and weights; clamped to the last block, a
  // harmless reload) go out first; scheduling barriers keep them above the
  // math and the LDS store of block b + 1 (loaded kRing - 2 steps ago) below
  // it.
#define MOE_PF_STEP(U, B)                                                                  \
  do {                                                                                     \
    const int b_ = (B);                                                                    \
    const int bl_ = b_ + kRing - 1 < nb ? b_ + kRing - 1 : nb - 1;                         \
    MOE_PF_ALOAD(((U) + kRing - 1) % kRing, bl_);                                          \
    MOE_PF_WLOAD(((U) + kRing - 1) % kRing, bl_);                                          \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    const uint8_t* sB = smem + (b_ & 1) * kStage + r * kLdsRow + kq * 16;                  \
    const float* sa_b = sa_lds + b_ * kSaStride + r;                                       \
    const float sw0 = swf0[b_], sw1 = swf1[b_];                                            \
    /* products of operand i are promoted while those of i + 1 run */                      \
    v8i bx = load_v8i_ksplit(sB);                                                          \
    v4f p0 = mfma_f8_16x16x128(wr[U][0], bx);                                              \
    v4f p1 = mfma_f8_16x16x128(wr[U][1], bx);                                              \
    _Pragma("unroll") for (int i = 0; i < 8; ++i) {                                        \
      v4f n0, n1;                                                                          \
      if (i < 7) {                                                                         \
        bx = load_v8i_ksplit(sB + (i + 1) * 16 * kLdsRow);                                 \
        n0 = mfma_f8_16x16x128(wr[U][0], bx);                                              \
        n1 = mfma_f8_16x16x128(wr[U][1], bx);                                              \
      }                                                                                    \
      const float sa = sa_b[i * 16];                                                       \
      const float s0 = sa * sw0, s1 = sa * sw1;                                            \
      _Pragma("unroll") for (int q = 0; q < 4; ++q) {                                      \
        acc[0][i][q] += p0[q] * s0;                                                        \
        acc[1][i][q] += p1[q] * s1;                                                        \
      }                                                                                    \
      if (i < 7) { p0 = n0; p1 = n1; }                                                     \
    }                                                                                      \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    MOE_PF_ASTORE(((U) + 1) % kRing, (b_ + 1) & 1);                                        \
    __syncthreads();                                                                       \
  } while (0)

#pragma unroll
  for (int s = 0; s < kRing - 1; ++s) {
    MOE_PF_ALOAD(s, s < nb ? s : nb - 1);
    MOE_PF_WLOAD(s, s < nb ? s : nb - 1);
  }
  MOE_PF_ASTORE(0, 0);
  __syncthreads();

  int b0 = 0;
  for (; b0 + kRing <= nb; b0 += kRing) {
    MOE_PF_STEP(0, b0);
    MOE_PF_STEP(1, b0 + 1);
    MOE_PF_STEP(2, b0 + 2);
    MOE_PF_STEP(3, b0 + 3);
  }
  if (b0 < nb) MOE_PF_STEP(0, b0);
  if (b0 + 1 < nb) MOE_PF_STEP(1, b0 + 1);
  if (b0 + 2 < nb) MOE_PF_STEP(2, b0 + 2);
#undef MOE_PF_WLOAD
#undef MOE_PF_ALOAD
#undef MOE_PF_ASTORE
#undef MOE_PF_STEP

  if (!GATEUP) {
    // y[m0 + t][nt*256 + 32w + 16f + 4kq + q] for expert row t = 16i + r.
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int t = i * 16 + r;
      if (t < mc) {
        float* dst = p.y + (int64_t)(m0 + t) * p.N + nt * kBN + wave * 32 + kq * 4;
#pragma unroll
        for (int f = 0; f < 2; ++f) *reinterpret_cast<v4f*>(dst + f * 16) = acc[f][i];
      }
    }
    return;
  }

  // GATEUP epilogue: h = SiLU(G) * U for channels 16w + 4kq + q of rows
  // t = 16i + r; per-row amax over the lane's 4 channels, the 4 lanes of
  // the row (kq) and the 8 waves.
  float h[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float mx = 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      h[i][q] = silu_mul(acc[0][i][q], acc[1][i][q]);
      mx = fmaxf(mx, fabsf(h[i][q]));
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (kq == 0) rowmax[wave][i * 16 + r] = mx;
  }
  __syncthreads();
  uint8_t* qtile = smem;  // [kBM][kLdsRow], the K-loop buffers are free now
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int t = i * 16 + r;
    float amax = rowmax[0][t];
#pragma unroll
    for (int w = 1; w < 8; ++w) amax = fmaxf(amax, rowmax[w][t]);
    const float s = amax / kE4M3Max;
    uint32_t packed = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) packed |= quantize_e4m3(h[i][q], s) << (8 * q);
    *reinterpret_cast<uint32_t*>(qtile + t * kLdsRow + wave * 16 + kq * 4) = packed;
    if (wave == 0 && kq == 0 && t < mc) p.sh[(int64_t)(m0 + t) * (p.N / kBlock) + nt] = s;
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
  if ((int64_t)a.N * a.K > 0x7fffffff)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: one expert matrix (%d x %d) exceeds 2 GiB", a.N, a.K);
  const size_t lds = 2 * (size_t)kStage + sizeof(float) * ((size_t)kSaStride + 2) * (a.K / kBlock);
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
