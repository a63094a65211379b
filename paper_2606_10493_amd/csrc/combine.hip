// Router-weighted combine: the k expert rows of a token are summed with the
// router weights in fp32, in slot order from +0.0, then rounded once to bf16
// (the paper's router-weighted F32 accumulation followed by conversion back
// to the hidden type).  Products and sums are rounded separately (FMA
// contraction is switched off in combine8_batched), which is the exact order of the
// definition, so the result is bit-identical to it for given rows.
//
// Memory bound: k * 4 bytes read + 2 bytes written per output element.
// Thread = 8 consecutive outputs (two 16-byte loads per slot, one 16-byte
// store); workgroup = 128 threads = 1024 outputs of one token.  Measured at
// 5.1 TB/s on 8192 tokens x 8 slots (1.88 GB of rows read).
#include "common.h"

namespace moe {
namespace {

// Slots in batches of 8: the batch's row indices and weights are loaded
// first, then its 8 rows (16 loads in flight per thread), then the products
// are added in slot order.  A slot past k reloads slot k-1 and is not
// added.  Same arithmetic and order as combine8_of (the fused decode
// kernel's combine), so the same bits.
__device__ __forceinline__ uint4 combine8_batched(const float* __restrict__ y, const int32_t* __restrict__ dest,
                                                  const float* __restrict__ w, int k, int H, int64_t t, int n) {
#pragma clang fp contract(off)
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
  for (int j0 = 0; j0 < k; j0 += 8) {
    int64_t p[8];
    float wj[8], v[8][8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = min(j0 + u, k - 1);
      p[u] = dest[t * k + j];
      wj[u] = w[t * k + j];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) load8_f32(y + p[u] * H + n, v[u]);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (j0 + u < k) {
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = acc[i] + wj[u] * v[u][i];
      }
  }
  uint4 o;
  o.x = (uint32_t)f32_to_bf16_rne(acc[0]) | ((uint32_t)f32_to_bf16_rne(acc[1]) << 16);
  o.y = (uint32_t)f32_to_bf16_rne(acc[2]) | ((uint32_t)f32_to_bf16_rne(acc[3]) << 16);
  o.z = (uint32_t)f32_to_bf16_rne(acc[4]) | ((uint32_t)f32_to_bf16_rne(acc[5]) << 16);
  o.w = (uint32_t)f32_to_bf16_rne(acc[6]) | ((uint32_t)f32_to_bf16_rne(acc[7]) << 16);
  return o;
}

__global__ __launch_bounds__(128) void combine_kernel(const float* __restrict__ y, const int32_t* __restrict__ dest,
                                                      const float* __restrict__ w, int k, int H, int blocks_per_tok,
                                                      uint16_t* __restrict__ out) {
  const int64_t t = blockIdx.x / blocks_per_tok;
  const int n = ((int)(blockIdx.x - t * blocks_per_tok) * 128 + (int)threadIdx.x) * 8;
  if (n >= H) return;
  *reinterpret_cast<uint4*>(out + t * H + n) = combine8_batched(y, dest, w, k, H, t, n);
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status_t moe_combine(const float* y_rows, const int32_t* dest_row, const float* topk_w, int32_t T,
                                    int32_t k, int32_t H, uint16_t* out_bf16, hipStream_t stream) {
  if (T < 0 || k < 1 || H <= 0) return fail(MOE_ERR_INVALID_ARG, "moe_combine: T=%d k=%d H=%d", T, k, H);
  if (H % kBlock) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_combine: H=%d not a multiple of 128", H);
  if (T == 0) return MOE_OK;
  if (!y_rows || !dest_row || !topk_w || !out_bf16) return fail(MOE_ERR_INVALID_ARG, "moe_combine: null pointer");
  if (!aligned(y_rows, 16) || !aligned(out_bf16, 16))
    return fail(MOE_ERR_INVALID_ARG, "moe_combine: misaligned pointer");
  const int bpt = (H + 1023) / 1024;
  const int64_t blocks = (int64_t)T * bpt;
  if (blocks > 0x7fffffff) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_combine: too many tokens");
  MOE_LAUNCH("combine", combine_kernel, dim3((unsigned)blocks), dim3(128), 0, stream, y_rows, dest_row, topk_w, k, H,
                     bpt, out_bf16);
  return check_launch("moe_combine");
}
