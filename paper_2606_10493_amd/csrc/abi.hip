// C ABI glue: status strings, per-thread error detail, workspace sizing and
// the regime dispatch of moe_expert_ffn.
#include <stdarg.h>
#include <stdio.h>

#include "common.h"

namespace moe {

static thread_local char g_last_error[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
}

moe_status_t fail(moe_status_t st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

moe_status_t check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(MOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return MOE_OK;
}

moe_status_t run_ffn_decode(const moe_dims_t& d, int32_t T, const uint8_t* qx, const float* sx,
                            const int32_t* offsets, const int32_t* sorted_src, const uint8_t* w_gate,
                            const float* s_gate, const uint8_t* w_up, const float* s_up, const uint8_t* w_down,
                            const float* s_down, float* y_rows, float* h, uint8_t* qh, float* sh,
                            hipStream_t stream);

moe_status_t run_ffn_decode_gateup(const moe_dims_t& d, int32_t T, const uint8_t* qx, const float* sx,
                                   const int32_t* offsets, const int32_t* sorted_src, const uint8_t* w_gate,
                                   const float* s_gate, const uint8_t* w_up, const float* s_up, float* h,
                                   hipStream_t stream);

bool decode_one_token_fits(const moe_dims_t& d);
moe_status_t run_ffn_decode_gateup_one_token(const moe_dims_t& d, const uint16_t* x, const int32_t* topk_ids,
                                             int32_t* dev_status, const uint8_t* w_gate, const float* s_gate,
                                             const uint8_t* w_up, const float* s_up, float* h, hipStream_t stream);

bool decode_down_combine_fits(const moe_dims_t& d, int32_t T);
moe_status_t run_ffn_decode_down_combine(const moe_dims_t& d, int32_t T, const float* h, const int32_t* offsets,
                                         const uint8_t* w_down, const float* s_down, const int32_t* dest_row,
                                         const float* topk_w, uint16_t* out, hipStream_t stream);
moe_status_t run_ffn_decode_down_combine_one_token(const moe_dims_t& d, const float* h, const int32_t* topk_ids,
                                                   const uint8_t* w_down, const float* s_down, const float* topk_w,
                                                   uint16_t* out, hipStream_t stream);

moe_status_t launch_layer_prologue(const uint16_t* x, int32_t T, int32_t H, const int32_t* topk_ids, int32_t k,
                                   int32_t E, uint8_t* qx, float* sx, int32_t* offsets, int32_t* sorted_src,
                                   int32_t* dest_row, int32_t* dev_status, hipStream_t stream);

moe_status_t run_ffn_prefill(const moe_dims_t& d, int32_t T, const uint8_t* qx, const float* sx,
                             const int32_t* offsets, const int32_t* sorted_src, const uint8_t* w_gate,
                             const float* s_gate, const uint8_t* w_up, const float* s_up, const uint8_t* w_down,
                             const float* s_down, float* y_rows, uint8_t* qh, float* sh, int32_t* tiles,
                             hipStream_t stream);

size_t prefill_tile_workspace(const moe_dims_t& d, int32_t T);
moe_status_t prefill_shape_check(const moe_dims_t& d);
moe_status_t decode_shape_check(const moe_dims_t& d);

moe_status_t run_ffn_decode_w8a16(const moe_dims_t& d, int32_t T, const uint16_t* x, const int32_t* offsets,
                                  const int32_t* sorted_src, const uint8_t* w_gate, const float* s_gate,
                                  const uint8_t* w_up, const float* s_up, const uint8_t* w_down,
                                  const float* s_down, float* y_rows, uint16_t* h16, hipStream_t stream);

namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

moe_regime_t resolve(moe_regime_t r, int32_t T) {
  if (r == MOE_REGIME_AUTO) return T <= MOE_DECODE_MAX_TOKENS ? MOE_REGIME_DECODE : MOE_REGIME_PREFILL;
  return r;
}

moe_status_t check_dims(const moe_dims_t& d, const char* who) {
  if (d.hidden <= 0 || d.inter <= 0 || d.n_experts < 1 || d.n_experts > 1024 || d.topk < 1 || d.topk > 32 ||
      d.topk > d.n_experts)
    return fail(MOE_ERR_INVALID_ARG, "%s: dims H=%d I=%d E=%d k=%d", who, d.hidden, d.inter, d.n_experts, d.topk);
  if (d.hidden % kBlock || d.inter % kBlock)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "%s: H=%d, I=%d must be multiples of 128", who, d.hidden, d.inter);
  return MOE_OK;
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" const char* moe_status_string(moe_status_t s) {
  switch (s) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG";
    case MOE_ERR_UNSUPPORTED_SHAPE: return "MOE_ERR_UNSUPPORTED_SHAPE";
    case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE";
    case MOE_ERR_HIP: return "MOE_ERR_HIP";
  }
  return "MOE_ERR_UNKNOWN";
}

extern "C" const char* moe_last_error(void) { return g_last_error; }

extern "C" size_t moe_expert_ffn_workspace(moe_dims_t d, int32_t T, moe_regime_t regime) {
  if (T < 0 || d.hidden <= 0 || d.inter <= 0 || d.topk <= 0 || d.n_experts <= 0) return 0;
  const size_t R = (size_t)T * d.topk;
  const size_t qh = align256(R * d.inter);
  const size_t sh = align256(R * (d.inter / kBlock) * sizeof(float));
  if (resolve(regime, T) == MOE_REGIME_DECODE) return qh + sh + align256(R * d.inter * sizeof(float));
  return qh + sh + align256(prefill_tile_workspace(d, T));
}

extern "C" moe_status_t moe_expert_ffn(moe_dims_t d, int32_t T, moe_regime_t regime, const uint8_t* qx,
                                       const float* sx, const int32_t* expert_offsets, const int32_t* sorted_src,
                                       const uint8_t* w_gate, const float* s_gate, const uint8_t* w_up,
                                       const float* s_up, const uint8_t* w_down, const float* s_down, float* y_rows,
                                       void* ws, size_t ws_bytes, hipStream_t stream) {
  moe_status_t st = check_dims(d, "moe_expert_ffn");
  if (st != MOE_OK) return st;
  if (T < 0) return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn: T=%d", T);
  if (regime != MOE_REGIME_AUTO && regime != MOE_REGIME_DECODE && regime != MOE_REGIME_PREFILL)
    return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn: regime=%d", (int)regime);
  const moe_regime_t rg = resolve(regime, T);
  if (rg == MOE_REGIME_DECODE && T > MOE_DECODE_MAX_TOKENS)
    return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn: decode regime needs T <= %d (T=%d)", MOE_DECODE_MAX_TOKENS, T);
  if ((int64_t)T * d.topk > 0x7fffffff) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_expert_ffn: T*k overflows");
  if (T == 0) return MOE_OK;
  if (!qx || !sx || !expert_offsets || !sorted_src || !w_gate || !s_gate || !w_up || !s_up || !w_down || !s_down ||
      !y_rows)
    return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn: null pointer");
  if (!aligned(qx, 16) || !aligned(w_gate, 16) || !aligned(w_up, 16) || !aligned(w_down, 16) ||
      !aligned(y_rows, 16) || !aligned(sx, 4))
    return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn: misaligned pointer (16 bytes needed)");
  const size_t need = moe_expert_ffn_workspace(d, T, rg);
  if (!ws || ws_bytes < need)
    return fail(MOE_ERR_WORKSPACE, "moe_expert_ffn: workspace %zu bytes < %zu", ws_bytes, need);
  if (!aligned(ws, 256)) return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn: workspace must be 256-byte aligned");
  const size_t R = (size_t)T * d.topk;
  uint8_t* base = static_cast<uint8_t*>(ws);
  uint8_t* qh = base;
  float* sh = reinterpret_cast<float*>(base + align256(R * d.inter));
  uint8_t* rest = reinterpret_cast<uint8_t*>(sh) + align256(R * (d.inter / kBlock) * sizeof(float));
  if (rg == MOE_REGIME_DECODE)
    return run_ffn_decode(d, T, qx, sx, expert_offsets, sorted_src, w_gate, s_gate, w_up, s_up, w_down, s_down,
                          y_rows, reinterpret_cast<float*>(rest), qh, sh, stream);
  return run_ffn_prefill(d, T, qx, sx, expert_offsets, sorted_src, w_gate, s_gate, w_up, s_up, w_down, s_down, y_rows,
                         qh, sh, reinterpret_cast<int32_t*>(rest), stream);
}

extern "C" size_t moe_expert_ffn_w8a16_workspace(moe_dims_t d, int32_t T) {
  if (T < 0 || d.inter <= 0 || d.topk <= 0) return 0;
  return align256((size_t)T * d.topk * d.inter * sizeof(uint16_t));
}

extern "C" moe_status_t moe_expert_ffn_w8a16(moe_dims_t d, int32_t T, const uint16_t* x_bf16,
                                             const int32_t* expert_offsets, const int32_t* sorted_src,
                                             const uint8_t* w_gate, const float* s_gate, const uint8_t* w_up,
                                             const float* s_up, const uint8_t* w_down, const float* s_down,
                                             float* y_rows, void* ws, size_t ws_bytes, hipStream_t stream) {
  moe_status_t st = check_dims(d, "moe_expert_ffn_w8a16");
  if (st != MOE_OK) return st;
  if (T < 0 || T > MOE_DECODE_MAX_TOKENS)
    return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn_w8a16: decode regime needs 0 <= T <= %d (T=%d)",
                MOE_DECODE_MAX_TOKENS, T);
  if (T == 0) return MOE_OK;
  if (!x_bf16 || !expert_offsets || !sorted_src || !w_gate || !s_gate || !w_up || !s_up || !w_down || !s_down ||
      !y_rows)
    return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn_w8a16: null pointer");
  if (!aligned(x_bf16, 16) || !aligned(w_gate, 16) || !aligned(w_up, 16) || !aligned(w_down, 16) ||
      !aligned(y_rows, 16))
    return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn_w8a16: misaligned pointer (16 bytes needed)");
  const size_t need = moe_expert_ffn_w8a16_workspace(d, T);
  if (!ws || ws_bytes < need)
    return fail(MOE_ERR_WORKSPACE, "moe_expert_ffn_w8a16: workspace %zu bytes < %zu", ws_bytes, need);
  if (!aligned(ws, 256)) return fail(MOE_ERR_INVALID_ARG, "moe_expert_ffn_w8a16: workspace must be 256-byte aligned");
  return run_ffn_decode_w8a16(d, T, x_bf16, expert_offsets, sorted_src, w_gate, s_gate, w_up, s_up, w_down, s_down,
                              y_rows, static_cast<uint16_t*>(ws), stream);
}

// ---------------------------------------------------------------- whole layer

namespace {

// moe_ffn_layer workspace: the intermediate tensors of the layer, each
// 256-byte aligned, then the permutation and expert-FFN workspaces.
struct LayerLayout {
  size_t qx, sx, offsets, sorted_src, dest_row, y, perm, ffn, total;
};

LayerLayout layer_layout(const moe_dims_t& d, int32_t T, moe_regime_t rg) {
  LayerLayout L{};
  const size_t R = (size_t)T * d.topk;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  L.qx = take((size_t)T * d.hidden);
  L.sx = take((size_t)T * (d.hidden / kBlock) * sizeof(float));
  L.offsets = take((size_t)(d.n_experts + 1) * sizeof(int32_t));
  L.sorted_src = take(R * sizeof(int32_t));
  L.dest_row = take(R * sizeof(int32_t));
  L.y = take(R * d.hidden * sizeof(float));
  L.perm = take(moe_permute_workspace(T, d.topk, d.n_experts));
  L.ffn = take(moe_expert_ffn_workspace(d, T, rg));
  L.total = off;
  return L;
}

}  // namespace

extern "C" size_t moe_ffn_layer_workspace(moe_dims_t d, int32_t T, moe_regime_t regime) {
  if (check_dims(d, "moe_ffn_layer_workspace") != MOE_OK || T < 0) return 0;
  return layer_layout(d, T, resolve(regime, T)).total;
}

extern "C" moe_status_t moe_ffn_layer(moe_dims_t d, int32_t T, moe_regime_t regime, const uint16_t* x_bf16,
                                      const int32_t* topk_ids, const float* topk_w, const uint8_t* w_gate,
                                      const float* s_gate, const uint8_t* w_up, const float* s_up,
                                      const uint8_t* w_down, const float* s_down, uint16_t* out_bf16,
                                      int32_t* dev_status, void* ws, size_t ws_bytes, hipStream_t stream) {
  moe_status_t st = check_dims(d, "moe_ffn_layer");
  if (st != MOE_OK) return st;
  if (T < 0) return fail(MOE_ERR_INVALID_ARG, "moe_ffn_layer: T=%d", T);
  if (regime != MOE_REGIME_AUTO && regime != MOE_REGIME_DECODE && regime != MOE_REGIME_PREFILL)
    return fail(MOE_ERR_INVALID_ARG, "moe_ffn_layer: regime=%d", (int)regime);
  const moe_regime_t rg = resolve(regime, T);
  if (rg == MOE_REGIME_DECODE && T > MOE_DECODE_MAX_TOKENS)
    return fail(MOE_ERR_INVALID_ARG, "moe_ffn_layer: decode regime needs T <= %d (T=%d)", MOE_DECODE_MAX_TOKENS, T);
  if ((int64_t)T * d.topk > 0x7fffffff) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_ffn_layer: T*k overflows");
  if (T == 0) return MOE_OK;
  if (!x_bf16 || !topk_ids || !topk_w || !w_gate || !s_gate || !w_up || !s_up || !w_down || !s_down || !out_bf16)
    return fail(MOE_ERR_INVALID_ARG, "moe_ffn_layer: null pointer");
  if (!aligned(x_bf16, 16) || !aligned(out_bf16, 16) || !aligned(w_gate, 16) || !aligned(w_up, 16) ||
      !aligned(w_down, 16))
    return fail(MOE_ERR_INVALID_ARG, "moe_ffn_layer: misaligned pointer (16 bytes needed)");
  st = rg == MOE_REGIME_DECODE ? decode_shape_check(d) : prefill_shape_check(d);
  if (st != MOE_OK) return st;
  const LayerLayout L = layer_layout(d, T, rg);
  if (!ws || ws_bytes < L.total)
    return fail(MOE_ERR_WORKSPACE, "moe_ffn_layer: workspace %zu bytes < %zu", ws_bytes, L.total);
  if (!aligned(ws, 256)) return fail(MOE_ERR_INVALID_ARG, "moe_ffn_layer: workspace must be 256-byte aligned");
  uint8_t* b = static_cast<uint8_t*>(ws);
  uint8_t* qx = b + L.qx;
  float* sx = reinterpret_cast<float*>(b + L.sx);
  int32_t* offsets = reinterpret_cast<int32_t*>(b + L.offsets);
  int32_t* sorted_src = reinterpret_cast<int32_t*>(b + L.sorted_src);
  int32_t* dest_row = reinterpret_cast<int32_t*>(b + L.dest_row);
  float* y = reinterpret_cast<float*>(b + L.y);
  const size_t R = (size_t)T * d.topk;

  if (rg == MOE_REGIME_DECODE && T == 1 && decode_down_combine_fits(d, T) && decode_one_token_fits(d)) {
    // One token: two launches and no prologue.  Gate/up quantizes the row
    // and reads the expert ids itself (row j of h is slot j); the down
    // projection and the combine follow in one launch.  The results are
    // bit-identical to the sorted path below.
    float* h = reinterpret_cast<float*>(b + L.ffn);
    st = run_ffn_decode_gateup_one_token(d, x_bf16, topk_ids, dev_status, w_gate, s_gate, w_up, s_up, h, stream);
    if (st != MOE_OK) return st;
    return run_ffn_decode_down_combine_one_token(d, h, topk_ids, w_down, s_down, topk_w, out_bf16, stream);
  }

  // Quantize and sort: one launch for a single chunk of tokens.
  if (T <= 256) {
    st = launch_layer_prologue(x_bf16, T, d.hidden, topk_ids, d.topk, d.n_experts, qx, sx, offsets, sorted_src,
                               dest_row, dev_status, stream);
  } else {
    st = moe_quant_act(x_bf16, T, d.hidden, qx, sx, stream);
    if (st == MOE_OK)
      st = moe_permute(topk_ids, T, d.topk, d.n_experts, offsets, sorted_src, dest_row, dev_status, b + L.perm,
                       moe_permute_workspace(T, d.topk, d.n_experts), stream);
  }
  if (st != MOE_OK) return st;

  if (rg == MOE_REGIME_DECODE && decode_down_combine_fits(d, T)) {
    // Gate/up, then the down projection and the combine in one launch (the
    // fp32 expert rows stay in LDS).
    uint8_t* qh = b + L.ffn;
    float* sh = reinterpret_cast<float*>(qh + align256(R * d.inter));
    float* h = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(sh) + align256(R * (d.inter / kBlock) * sizeof(float)));
    st = run_ffn_decode_gateup(d, T, qx, sx, offsets, sorted_src, w_gate, s_gate, w_up, s_up, h, stream);
    if (st != MOE_OK) return st;
    return run_ffn_decode_down_combine(d, T, h, offsets, w_down, s_down, dest_row, topk_w, out_bf16, stream);
  }
  st = moe_expert_ffn(d, T, rg, qx, sx, offsets, sorted_src, w_gate, s_gate, w_up, s_up, w_down, s_down, y,
                      b + L.ffn, moe_expert_ffn_workspace(d, T, rg), stream);
  if (st != MOE_OK) return st;
  return moe_combine(y, dest_row, topk_w, T, d.topk, d.hidden, out_bf16, stream);
}
