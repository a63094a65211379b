// Block quantization to FP8 e4m3 (FP8 Block Scaling Format; 128-element scale
// blocks as in the FP8 GEMV kernel's scale-block loop).
//
// Activations / h: one scale per row per 128 consecutive columns.  A group of
// 16 lanes owns one 128-column block (8 elements per lane, one 16-byte load
// of bf16 or two of fp32), reduces |x| with cross-lane xor shuffles, divides
// and encodes.  Memory bound: 2 (bf16) or 4 (fp32) bytes read + 1 byte
// written per element, + 4 bytes per 128 elements.
//
// Weights: one scale per 128x128 block; one 256-thread workgroup per block.
#include "common.h"

namespace moe {

namespace {

__device__ __forceinline__ uint2 encode8(const float (&v)[8], float s) {
  return make_uint2(quantize4_e4m3(v[0], v[1], v[2], v[3], s), quantize4_e4m3(v[4], v[5], v[6], v[7], s));
}

// grid: ceil(rows * cols/128 / 16) blocks of 256 threads; 16 groups per block.
template <typename InT>
__global__ __launch_bounds__(256) void quant_rows_kernel(const InT* __restrict__ x, int64_t n_groups,
                                                         int groups_per_row, uint8_t* __restrict__ q,
                                                         float* __restrict__ s) {
  const int64_t g = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  if (g >= n_groups) return;  // whole 16-lane groups leave together
  quant_row_group<InT>(x, g, threadIdx.x & 15, groups_per_row, q, s);
}

// One 256-thread workgroup per 128x128 block.  Thread t covers columns
// 8*(t%16) .. +7 of rows t/16 + 16*r, r = 0..7.
__global__ __launch_bounds__(256) void quant_weight_kernel(const float* __restrict__ w, int rows, int cols,
                                                           uint8_t* __restrict__ q, float* __restrict__ s) {
  const int nbc = cols / kBlock, nbr = rows / kBlock;
  const int64_t blk = blockIdx.x;
  const int64_t mat = blk / ((int64_t)nbr * nbc);
  const int rem = (int)(blk - mat * nbr * nbc);
  const int br = rem / nbc, bc = rem % nbc;
  const int t = threadIdx.x;
  const int c = bc * kBlock + (t & 15) * 8;
  const int64_t base = mat * (int64_t)rows * cols;
  float v[8][8];
  float amax = 0.0f;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int row = br * kBlock + (t >> 4) + 16 * r;
    load8_f32(w + base + (int64_t)row * cols + c, v[r]);
#pragma unroll
    for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[r][i]));
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) amax = fmaxf(amax, __shfl_xor(amax, m, 64));
  __shared__ float wave_max[4];
  if ((t & 63) == 0) wave_max[t >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(wave_max[0], wave_max[1]), fmaxf(wave_max[2], wave_max[3]));
  const float sc = amax / kE4M3Max;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int row = br * kBlock + (t >> 4) + 16 * r;
    *reinterpret_cast<uint2*>(q + base + (int64_t)row * cols + c) = encode8(v[r], sc);
  }
  if (t == 0) s[blk] = sc;
}

template <typename InT>
moe_status_t quant_rows(const InT* x, int32_t rows, int32_t cols, uint8_t* q, float* s, hipStream_t stream,
                        const char* name) {
  if (rows < 0 || cols <= 0) return fail(MOE_ERR_INVALID_ARG, "%s: rows=%d cols=%d", name, rows, cols);
  if (cols % kBlock) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "%s: cols=%d not a multiple of 128", name, cols);
  if (rows == 0) return MOE_OK;
  if (!x || !q || !s) return fail(MOE_ERR_INVALID_ARG, "%s: null pointer", name);
  if (!aligned(x, 16) || !aligned(q, 8) || !aligned(s, 4))
    return fail(MOE_ERR_INVALID_ARG, "%s: misaligned pointer", name);
  const int gpr = cols / kBlock;
  const int64_t n_groups = (int64_t)rows * gpr;
  const int64_t blocks = (n_groups + 15) / 16;
  MOE_LAUNCH(name, quant_rows_kernel<InT>, dim3((unsigned)blocks), dim3(256), 0, stream, x, n_groups, gpr, q, s);
  return check_launch(name);
}

// Row-major e4m3 [total_rows, cols] -> packed operand tiles (the layout is
// described with packed_lane_offset).  One thread moves one 16-byte chunk:
// output chunk c of tile c / 128 holds half h = (c >> 6) & 1, kq = 2 *
// ((c >> 4) & 1) + ((c >> 5) & 1), row r = c & 15 of the tile.
__global__ __launch_bounds__(256) void pack_weight_kernel(const uint8_t* __restrict__ q, int64_t chunks, int cols,
                                                          uint8_t* __restrict__ out) {
  const int nkb = cols / kBlock;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < chunks; c += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(c & 15), h = (int)((c >> 6) & 1);
    const int kq = 2 * (int)((c >> 4) & 1) + (int)((c >> 5) & 1);
    const int64_t tile = c >> 7;
    const int64_t g = tile / nkb;
    const int b = (int)(tile - g * nkb);
    const int64_t row = g * 16 + r;
    const int64_t col = (int64_t)b * kBlock + h * 64 + kq * 16;
    *reinterpret_cast<uint4*>(out + c * 16) = *reinterpret_cast<const uint4*>(q + row * cols + col);
  }
}

}  // namespace

}  // namespace moe

using namespace moe;

extern "C" moe_status_t moe_quant_act(const uint16_t* x_bf16, int32_t rows, int32_t cols, uint8_t* q, float* s,
                                      hipStream_t stream) {
  return quant_rows<uint16_t>(x_bf16, rows, cols, q, s, stream, "moe_quant_act");
}

extern "C" moe_status_t moe_quant_rows_f32(const float* x, int32_t rows, int32_t cols, uint8_t* q, float* s,
                                           hipStream_t stream) {
  return quant_rows<float>(x, rows, cols, q, s, stream, "moe_quant_rows_f32");
}

extern "C" moe_status_t moe_quant_weight(const float* w, int32_t n_mats, int32_t rows, int32_t cols, uint8_t* q,
                                         float* s, hipStream_t stream) {
  if (n_mats < 0 || rows <= 0 || cols <= 0)
    return fail(MOE_ERR_INVALID_ARG, "moe_quant_weight: n_mats=%d rows=%d cols=%d", n_mats, rows, cols);
  if (rows % kBlock || cols % kBlock)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_quant_weight: %dx%d not multiples of 128", rows, cols);
  if (n_mats == 0) return MOE_OK;
  if (!w || !q || !s) return fail(MOE_ERR_INVALID_ARG, "moe_quant_weight: null pointer");
  if (!aligned(w, 16) || !aligned(q, 8) || !aligned(s, 4))
    return fail(MOE_ERR_INVALID_ARG, "moe_quant_weight: misaligned pointer");
  const int64_t blocks = (int64_t)n_mats * (rows / kBlock) * (cols / kBlock);
  if (blocks > 0x7fffffff) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_quant_weight: too many blocks");
  MOE_LAUNCH("quant_weight", quant_weight_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, w, rows, cols, q, s);
  return check_launch("moe_quant_weight");
}

extern "C" moe_status_t moe_pack_weight(const uint8_t* q, int32_t n_mats, int32_t rows, int32_t cols,
                                        uint8_t* packed, hipStream_t stream) {
  if (n_mats < 0 || rows <= 0 || cols <= 0)
    return fail(MOE_ERR_INVALID_ARG, "moe_pack_weight: n_mats=%d rows=%d cols=%d", n_mats, rows, cols);
  if (rows % 16 || cols % kBlock)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_pack_weight: %dx%d needs rows %% 16 == 0 and cols %% 128 == 0", rows, cols);
  if (n_mats == 0) return MOE_OK;
  if (!q || !packed) return fail(MOE_ERR_INVALID_ARG, "moe_pack_weight: null pointer");
  if (q == packed) return fail(MOE_ERR_INVALID_ARG, "moe_pack_weight: packing in place is not supported");
  if (!aligned(q, 16) || !aligned(packed, 16)) return fail(MOE_ERR_INVALID_ARG, "moe_pack_weight: misaligned pointer");
  const int64_t chunks = (int64_t)n_mats * rows * (cols / 16);
  int64_t grid = (chunks + 255) / 256;
  if (grid > 65536) grid = 65536;
  MOE_LAUNCH("pack_weight", pack_weight_kernel, dim3((unsigned)grid), dim3(256), 0, stream, q, chunks, cols, packed);
  return check_launch("moe_pack_weight");
}
