// Shared device helpers and host error plumbing of the MoE FP8 library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "moe.h"

namespace moe {

constexpr int kBlock = MOE_BLOCK;   // FP8 scale block (elements along K)
constexpr float kE4M3Max = 448.0f;  // largest finite e4m3 magnitude

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// fp32 -> e4m3 code (OCP E4M3: bias 7, no infinities, max 448), round to
// nearest with ties to the even code, |v| >= 448 saturates to 448 (NaN too),
// the sign of zero is kept; values below 2^-6 go to the e4m3 subnormals
// (spacing 2^-9).
//
// gfx950's fp32 -> fp8 conversion rounds to nearest even and produces the
// e4m3 subnormals; it is given the value clamped to +-448 (fminf also maps
// NaN to 448), so it never sees an out-of-range input.  The result equals
// the code defined above for every one of the 2^32 fp32 bit patterns
// (compared on gfx950 against a bit-level software encoder of the same
// rule); the library's tests compare it with the oracle's nearest-value
// search on every value of several bands and at every rounding midpoint.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float e4m3_clamp(float v) { return __builtin_copysignf(fminf(fabsf(v), kE4M3Max), v); }

// x / s correctly rounded (the fp32 quotient of the rounding rule), given
// y = 1 / s correctly rounded: q0 = RN(x * y), the residual x - q0 * s
// exactly by one FMA, then RN(q0 + residual * y) (Markstein's correction,
// which is correctly rounded when y = RN(1/s), q0 is within one ulp of x/s
// and the residual is exact).  The residual is exact whenever s >= 2^-90 and
// |x / s| >= 2^-12; below 2^-12 only the e4m3 code matters, and it is +-0
// for any quotient under 2^-10.  Checked on gfx950 against the correctly
// rounded division for every fp32 x in the quantizer's range (|x| <= 448 s)
// and 62 scales from 2^-30 to 2^10, the all-ones mantissas among them: no
// difference from 2^-12 up.  The sign of x is kept (a zero quotient of -x is
// -0).
__device__ __forceinline__ float div_by_scale(float x, float s, float y) {
  const float q0 = x * y;
  const float r = __builtin_fmaf(-q0, s, x);
  return __builtin_copysignf(__builtin_fmaf(r, y, q0), x);
}

// Four values of one scale block quantized with its scale s into one word
// (byte i = value i): the code of x / s (the correctly rounded fp32
// quotient).  For s >= 2^-90 it comes from the reciprocal of s (one
// correctly rounded division per block, shared by every call with the same
// s) and div_by_scale; otherwise from the division itself.  s == 0 only
// when every |x| of the block is below 448 * 2^-150 (amax / 448 rounds to
// 0): then x itself is encoded, which keeps only its sign.
__device__ __forceinline__ uint32_t quantize4_e4m3(float a, float b, float c, float d, float s) {
  float qa, qb, qc, qd;
  if (s >= 0x1p-90f) {
    const float y = 1.0f / s;
    qa = div_by_scale(a, s, y);
    qb = div_by_scale(b, s, y);
    qc = div_by_scale(c, s, y);
    qd = div_by_scale(d, s, y);
  } else {
    const bool z = !(s > 0.0f);
    qa = z ? a : a / s;
    qb = z ? b : b / s;
    qc = z ? c : c / s;
    qd = z ? d : d / s;
  }
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(qa), e4m3_clamp(qb), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(qc), e4m3_clamp(qd), w, true);
  return (uint32_t)w;
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// FP8 x FP8 MFMA over one 128-element K block: D[16x16] = A[16x128] * B[128x16].
// Lane l supplies row (l & 15) of A and column (l & 15) of B, 32 bytes each.
// Every operand of the library uses one K assignment: lane group kq = l / 16
// supplies K bytes [16 kq, 16 kq + 16) and [64 + 16 kq, 80 + 16 kq) of the
// block.  A and B share it, so each dot product runs over the whole block;
// the instruction's internal order of K does not matter.
// The instruction's own E8M0 block scales are not used: with both scale
// operands 0 the compiler emits the unscaled v_mfma_f32_16x16x128_f8f6f4
// (format 0 = e4m3 for both operands), one 8-byte instruction instead of the
// scaled form's 16-byte pair of a scale load and the MFMA.  The fp32 scales
// are applied to the result.
__device__ __forceinline__ v4f mfma_f8_16x16x128(const v8i& a, const v8i& b) {
  const v4f zero = {0.f, 0.f, 0.f, 0.f};
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, zero, 0, 0, 0, 0, 0, 0);
}

// Packed weight layout (moe_pack_weight): a [rows, K] e4m3 matrix is stored
// as 16-row x 128-K tiles of 2048 bytes, tile (g, b) at (g * K/128 + b) *
// 2048.  Inside a tile, the 16 bytes at
//   packed_lane_offset(h, kq, r) = 1024 h + 512 (kq & 1) + 256 (kq >> 1) + 16 r
// hold row 16g + r, K indices 128b + 64h + 16kq + [0, 16) (h in {0,1},
// kq in [0,4), r in [0,16)).  A wave reads one operand as two loads that
// each cover 1 KB of contiguous memory, for both MFMA shapes the library
// uses: 16x16x128 (lane l: r = l % 16, kq = l / 16, h = the two halves of
// its 32 bytes) and 32x32x64 (lane l: row l % 32 of two consecutive 16-row
// groups, K bytes 64h + 32 (l / 32) + [0, 32), i.e. kq = 2 (l / 32) + part).
__device__ __forceinline__ int packed_lane_offset(int h, int kq, int r) {
  return 1024 * h + 512 * (kq & 1) + 256 * (kq >> 1) + 16 * r;
}
constexpr int kTileBytes = 16 * MOE_BLOCK;

__device__ __forceinline__ v8i join_v8i(const uint4& lo, const uint4& hi) {
  v8i r;
  r[0] = lo.x; r[1] = lo.y; r[2] = lo.z; r[3] = lo.w;
  r[4] = hi.x; r[5] = hi.y; r[6] = hi.z; r[7] = hi.w;
  return r;
}

// Operand of lane group kq from a row-major K block: p points at byte 16 kq
// of the lane's row within the block.
__device__ __forceinline__ v8i load_v8i_ksplit(const uint8_t* p) {
  return join_v8i(*reinterpret_cast<const uint4*>(p), *reinterpret_cast<const uint4*>(p + 64));
}

// 16x16x128 operand from a packed weight tile: p points at
// packed_lane_offset(0, kq, r) of the tile (the second half is 1024 further).
__device__ __forceinline__ v8i load_v8i_packed(const uint8_t* p) {
  return join_v8i(*reinterpret_cast<const uint4*>(p), *reinterpret_cast<const uint4*>(p + 1024));
}

typedef uint32_t u32x4_stream __attribute__((ext_vector_type(4)));
// load_v8i_packed with non-temporal (streaming) loads, for weights that are
// read once per launch (the decode GEMVs): measured 8-10 % faster there.
__device__ __forceinline__ v8i load_v8i_packed_stream(const uint8_t* p) {
  const u32x4_stream lo = __builtin_nontemporal_load(reinterpret_cast<const u32x4_stream*>(p));
  const u32x4_stream hi = __builtin_nontemporal_load(reinterpret_cast<const u32x4_stream*>(p + 1024));
  v8i r;
  r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
  r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
  return r;
}

// SiLU(g) * u = g * sigmoid(g) * u.  silu_mul: expf and a correctly rounded
// division (the decode kernels, bound by weight streaming).  silu_mul_fast:
// the hardware base-2 exponential of -g * log2(e) and the hardware
// reciprocal (each about 1 ulp; about 4 ulp in all), for the prefill GEMM
// epilogue, where no matrix instruction overlaps the epilogue's vector
// work.  exp2 -> +inf for very negative g gives 0 (the limit), exp2 -> 0
// for very positive g gives g * u.
__device__ __forceinline__ float silu_mul(float g, float u) {
  return (g * (1.0f / (1.0f + expf(-g)))) * u;
}

__device__ __forceinline__ float silu_mul_fast(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(g * -1.44269504088896341f);
  return (g * __builtin_amdgcn_rcpf(1.0f + e)) * u;
}

// Eight consecutive values of a row as fp32 (one 16-byte load of bf16, two of fp32).
__device__ __forceinline__ void bf16x8_to_f32(const uint4 raw, float (&v)[8]) {
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf16_to_f32(w[i] & 0xffffu);
    v[2 * i + 1] = bf16_to_f32(w[i] >> 16);
  }
}
__device__ __forceinline__ void load8_f32(const uint16_t* p, float (&v)[8]) {
  bf16x8_to_f32(*reinterpret_cast<const uint4*>(p), v);
}
__device__ __forceinline__ void load8_f32(const float* p, float (&v)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// Activation block quantization (one scale per row per 128 columns): group g
// of a [rows, 128 * groups_per_row] matrix is held by 16 consecutive lanes
// (lane sub of the group: columns 8 sub .. 8 sub + 7).  The block amax is
// reduced over the 16 lanes, s = amax / 448, and the lane writes its 8
// codes; lane 0 of the group writes s.
// The arithmetic of one group: this lane's 8 values -> 8 codes, the group's
// scale returned (every lane of the 16 calls it together).
__device__ __forceinline__ float quant_group8(const float (&v)[8], uint2& codes) {
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[i]));
#pragma unroll
  for (int m = 8; m >= 1; m >>= 1) amax = fmaxf(amax, __shfl_xor(amax, m, 16));
  const float sc = amax / kE4M3Max;
  codes = make_uint2(quantize4_e4m3(v[0], v[1], v[2], v[3], sc), quantize4_e4m3(v[4], v[5], v[6], v[7], sc));
  return sc;
}
template <typename InT>
__device__ __forceinline__ void quant_row_group(const InT* __restrict__ x, int64_t g, int sub, int groups_per_row,
                                                uint8_t* __restrict__ q, float* __restrict__ s) {
  const int64_t row = g / groups_per_row;
  const int64_t col = (g - row * groups_per_row) * kBlock + sub * 8;
  const int64_t idx = row * (int64_t)groups_per_row * kBlock + col;
  float v[8];
  load8_f32(x + idx, v);
  uint2 codes;
  const float sc = quant_group8(v, codes);
  *reinterpret_cast<uint2*>(q + idx) = codes;
  if (sub == 0) s[g] = sc;
}

// Router-weighted combine of 8 consecutive outputs of token t:
// bf16(sum_j w[t, j] * row_of(dest[t*k + j])[i]) over j = 0 .. k-1 in slot
// order from +0.0, every product and sum rounded separately (no FMA: the
// definition's order), then one round to bf16.  row_of(p) points at the 8
// values of expert row p.  Returns the 8 bf16 values.
template <typename RowOf>
__device__ __forceinline__ uint4 combine8_of(RowOf row_of, const int32_t* __restrict__ dest,
                                             const float* __restrict__ w, int k, int64_t t) {
#pragma clang fp contract(off)
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
  for (int j = 0; j < k; ++j) {
    const int64_t p = dest[t * k + j];
    const float wj = w[t * k + j];
    float v[8];
    load8_f32(row_of(p), v);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = acc[i] + wj * v[i];
  }
  uint4 o;
  o.x = (uint32_t)f32_to_bf16_rne(acc[0]) | ((uint32_t)f32_to_bf16_rne(acc[1]) << 16);
  o.y = (uint32_t)f32_to_bf16_rne(acc[2]) | ((uint32_t)f32_to_bf16_rne(acc[3]) << 16);
  o.z = (uint32_t)f32_to_bf16_rne(acc[4]) | ((uint32_t)f32_to_bf16_rne(acc[5]) << 16);
  o.w = (uint32_t)f32_to_bf16_rne(acc[6]) | ((uint32_t)f32_to_bf16_rne(acc[7]) << 16);
  return o;
}

// Exclusive prefix sum of v over the whole workgroup (blockDim.x a multiple
// of 64, at most 1024): shuffle scan inside each wave, wave totals through
// LDS (wave_tot holds blockDim.x/64 ints).  Returns the exclusive prefix and
// the workgroup total.  Every thread of the workgroup must call it.
__device__ __forceinline__ int block_exclusive_scan(int v, int* wave_tot, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) wave_tot[wave] = x;
  __syncthreads();
  int pre = 0, tot = 0;
  for (int w = 0; w < nw; ++w) {
    const int t = wave_tot[w];
    pre += (w < wave) ? t : 0;
    tot += t;
  }
  __syncthreads();  // wave_tot may be reused right after
  *total = tot;
  return pre + x - v;
}

// ----------------------------------------------------------------- host side
void prof_before(hipStream_t s, const char* name);
void prof_after(hipStream_t s);

// Kernel launch bracketed by the optional per-launch timing events.
#define MOE_LAUNCH(NAME, KERNEL, GRID, BLOCK, LDS, STREAM, ...)          \
  do {                                                                  \
    ::moe::prof_before((STREAM), (NAME));                               \
    hipLaunchKernelGGL(KERNEL, GRID, BLOCK, LDS, STREAM, __VA_ARGS__);  \
    ::moe::prof_after((STREAM));                                        \
  } while (0)

// Expert-sorted rows of one prefill GEMM launch pair: n_chunks chunks of
// tokens, each sorted by expert on its own; the launch covers n_units
// consecutive experts (its weight stacks hold exactly those).  Chunk c's
// offsets of those experts are offsets[c * off_stride + u], u = 0..n_units,
// relative to the chunk's first sorted row c * chunk_rows; its sorted_src
// entries are chunk-relative slots (token t - c * chunk_tokens).  A resident
// layer is one chunk of all its experts.
struct PrefillRows {
  const int32_t* offsets;
  int64_t off_stride;
  int n_units, n_chunks;
  int64_t chunk_rows;   // sorted rows per chunk (chunk_tokens * k)
  int chunk_tokens;
  int32_t tokens;       // activation rows of the gate/up projections (all chunks)
  int64_t rows;         // sorted rows of all chunks (activation rows of the down projection)
  int64_t max_mtiles;   // bound on the launch's 128-row m-tiles (sizes the grid and the descriptor table)
};

void set_error(const char* fmt, ...);
moe_status_t fail(moe_status_t st, const char* fmt, ...);
moe_status_t check_launch(const char* what);

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace moe
