/*
 * moe.h -- C ABI of the MI355X (gfx950) routed-expert FP8 MoE FFN library.
 *
 * One routed-expert MoE layer of a DeepSeek-V3-style model with FP8 e4m3
 * expert weights carrying fp32 scales per 128x128 weight block:
 *
 *   moe_quant_act   activations bf16 -> e4m3 per token per 128 channels
 *   moe_permute     top-k routing -> per-expert token lists
 *   moe_expert_ffn  per expert: gate and up projections, SiLU(gate)*up,
 *                   re-quantization, down projection (FP8 x FP8, fp32
 *                   accumulation, one scale per 128-K block)
 *   moe_combine     routing-weighted fp32 sum of the k expert rows -> bf16
 *   moe_ffn_streamed  the whole layer with the expert weights resident in
 *                   pinned host memory, copied block by block into a device
 *                   ring of expert slots on a copy stream while the compute
 *                   stream runs the experts whose weights have landed
 *
 * Conventions (all entry points):
 *   - Every pointer is owned by the caller.  "device" pointers are HIP device
 *     memory of the current device; "pinned host" pointers come from
 *     hipHostMalloc (or torch pin_memory).  The library never allocates,
 *     frees or synchronizes the host on these calls; all work is enqueued on
 *     the given stream(s) in order.
 *   - Layouts are row-major and contiguous.  Weights are [out, in] (the
 *     reduction dimension K contiguous); weight scales are
 *     [out/128, in/128]; activation scales are [rows, cols/128].
 *   - All feature dimensions must be multiples of 128 (the FP8 scale block),
 *     else MOE_ERR_UNSUPPORTED_SHAPE.  Argument errors are returned before
 *     anything is enqueued.  Launch failures return MOE_ERR_HIP (details in
 *     moe_last_error()).  Data errors found on the device (an expert id out
 *     of range or repeated within a token) are OR-ed into *dev_status.
 *   - Inputs must be finite.  Calls on distinct streams are thread-safe.
 */
#ifndef MOE_FP8_MI355X_H
#define MOE_FP8_MI355X_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_BLOCK 128

typedef enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = -1,
  MOE_ERR_UNSUPPORTED_SHAPE = -2,
  MOE_ERR_WORKSPACE = -3,
  MOE_ERR_HIP = -4
} moe_status_t;

/* Bits OR-ed into the optional device status word by moe_permute. */
#define MOE_DEV_BAD_EXPERT_ID 1  /* an id outside [0, n_experts) */
#define MOE_DEV_DUP_EXPERT_ID 2  /* the same id twice in one token's top-k */

/* Kernel family used by moe_expert_ffn.  AUTO picks DECODE for
 * tokens <= MOE_DECODE_MAX_TOKENS, else PREFILL; both compute the same
 * definition. */
typedef enum {
  MOE_REGIME_AUTO = 0,
  MOE_REGIME_DECODE = 1,  /* weight-streaming FP8 MFMA GEMV, tokens <= 64 */
  MOE_REGIME_PREFILL = 2  /* LDS-tiled block-scaled FP8 MFMA grouped GEMM */
} moe_regime_t;

#define MOE_DECODE_MAX_TOKENS 64

typedef struct {
  int32_t hidden;    /* H: model width, multiple of 128 */
  int32_t inter;     /* I: expert intermediate width, multiple of 128 */
  int32_t n_experts; /* E: routed experts in the layer, 1..1024 */
  int32_t topk;      /* k: experts per token, 1..min(E, 32) */
} moe_dims_t;

/* Human-readable name of a status code (static storage). */
const char* moe_status_string(moe_status_t status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* moe_last_error(void);

/*
 * Activation quantization (FP8 Block Scaling Format: activations are
 * quantized to FP8 before the FP8 GEMM; 128-element scale blocks as in the
 * Tiling and Scale-Block Optimizations of the FP8 GEMV kernel).
 *
 * For each row r and each block b of 128 consecutive columns:
 *   a = max |x[r, 128b .. 128b+127]|, s[r,b] = a / 448 (fp32, correctly
 *   rounded), q = e4m3 code nearest to x / s (correctly rounded fp32
 *   division; ties to the even code; |x/s| > 448 saturates to 448; the sign
 *   of zero is kept).  An all-zero block gives s = 0 and signed-zero codes.
 *
 * x_bf16: device [rows, cols] bf16 bit patterns.  q: device [rows, cols]
 * e4m3 codes.  s: device [rows, cols/128] fp32.  rows >= 0 (0 enqueues
 * nothing); cols a positive multiple of 128.
 */
moe_status_t moe_quant_act(const uint16_t* x_bf16, int32_t rows, int32_t cols,
                           uint8_t* q, float* s, hipStream_t stream);

/* Same rule over fp32 rows (used for the expert intermediate h). */
moe_status_t moe_quant_rows_f32(const float* x, int32_t rows, int32_t cols,
                                uint8_t* q, float* s, hipStream_t stream);

/*
 * Weight quantization to the DeepSeek-V3 FP8 storage format (FP8 Block
 * Scaling Format): per 128x128 block of each [rows, cols] matrix the same
 * rule as moe_quant_act with a = max over the 16384 block elements.
 *
 * w: device fp32 [n_mats, rows, cols].  q: device e4m3 [n_mats, rows, cols].
 * s: device fp32 [n_mats, rows/128, cols/128].  rows, cols multiples of 128.
 * This is offline weight preparation, not part of a layer call.
 */
moe_status_t moe_quant_weight(const float* w, int32_t n_mats, int32_t rows, int32_t cols,
                              uint8_t* q, float* s, hipStream_t stream);

/*
 * Weight packing into the operand-tile layout that moe_expert_ffn and
 * moe_ffn_streamed read (a storage order of the FP8 Block Scaling Format's
 * codes; the values and the 128x128 scales are unchanged).
 *
 * Each [rows, cols] matrix is cut into 16-row x 128-column tiles of 2048
 * bytes, stored row-group major: tile (g, b) starts at byte
 * (g * cols/128 + b) * 2048 of the matrix.  Inside a tile, the 16 bytes at
 *   1024*h + 512*(kq % 2) + 256*(kq / 2) + 16*r      (h in {0,1}, kq in [0,4), r in [0,16))
 * hold q[16g + r, 128b + 64h + 16kq + j] for j = 0..15: the orders in which
 * the 64 lanes of a wave feed a 16x16x128 and a 32x32x64 FP8 MFMA operand
 * both map to two fully contiguous 1 KB wave loads per operand.  A matrix
 * keeps its size (rows*cols bytes) and an expert's matrix stays contiguous.
 *
 * q: device e4m3 [n_mats, rows, cols] row-major (from moe_quant_weight).
 * packed: device, n_mats*rows*cols bytes, not overlapping q.  rows a
 * multiple of 16, cols a multiple of 128; both pointers 16-byte aligned.
 * Offline weight preparation, like moe_quant_weight.
 */
moe_status_t moe_pack_weight(const uint8_t* q, int32_t n_mats, int32_t rows, int32_t cols,
                             uint8_t* packed, hipStream_t stream);

/*
 * Token -> expert permutation (tokens are gated and sorted by expert into
 * per-expert token lists: Multi-GPU Parallelism and the standard EP
 * workflow of Distributed Stream-loading Prefill).
 *
 * Flat slot f = t*k + j holds expert topk_ids[t*k + j].  The slots are
 * stably sorted by expert id (ties by f):
 *   expert_offsets[e] = number of slots with id < e  (expert_offsets[E] = T*k)
 *   sorted_src[p]     = the slot f at sorted position p
 *   dest_row[f]       = the sorted position p of slot f
 * The result is unique, computed without order-dependent atomics, and
 * identical run to run.
 *
 * topk_ids: device int32 [T, k].  expert_offsets: device int32 [E+1].
 * sorted_src, dest_row: device int32 [T*k].  dev_status: device int32 or
 * NULL; bits MOE_DEV_* are OR-ed in when ids are bad (outputs are then
 * unspecified but every write stays in bounds).  ws: device workspace of at
 * least moe_permute_workspace(T, k, E) bytes.  T >= 0, 1 <= k <= min(E,32),
 * 1 <= E <= 1024.
 */
size_t moe_permute_workspace(int32_t T, int32_t k, int32_t E);
moe_status_t moe_permute(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                         int32_t* expert_offsets, int32_t* sorted_src, int32_t* dest_row,
                         int32_t* dev_status, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Routed expert FFN over the expert-sorted rows (Fine-grained CPU
 * Parallelism for MoE Inference: gate and up are independent, SiLU(gate)
 * times up is fused into stage one, then down; FP8 x FP8 GEMMs with fp32
 * accumulation and one fp32 scale per 128-K block).
 *
 * Row p (0 <= p < T*k) belongs to token t = sorted_src[p] / k and to the
 * expert e with expert_offsets[e] <= p < expert_offsets[e+1].  For each n:
 *   G[p,n] = sum_b (sx[t,b] * s_gate[e,n/128,b]) * sum_{i in b} qx[t,i] w_gate[e,n,i]
 *   U[p,n] likewise with w_up, s_up
 *   h = G * sigmoid(G) * U (fp32), quantized per row per 128 -> qh, sh
 *   y_rows[p,m] = sum_b (sh[p,b] * s_down[e,m/128,b]) * sum_{i in b} qh[p,i] w_down[e,m,i]
 *
 * qx: device e4m3 [T, H]; sx: device fp32 [T, H/128] (from moe_quant_act).
 * w_gate, w_up: device e4m3 [E, I, H]; s_gate, s_up: fp32 [E, I/128, H/128].
 * w_down: device e4m3 [E, H, I]; s_down: fp32 [E, H/128, I/128].
 * The three weight stacks are in the packed layout of moe_pack_weight
 * (the scales stay row-major).  The layout cannot be checked: row-major
 * (unpacked) stacks, as a checkpoint stores them, give undefined results.
 * y_rows: device fp32 [T*k, H] in expert-sorted order.
 * ws: device workspace of moe_expert_ffn_workspace(dims, T, regime) bytes.
 * regime: see moe_regime_t; DECODE requires T <= MOE_DECODE_MAX_TOKENS.
 * The PREFILL regime requires H % 256 == 0, max(H, I) <= 24576 and
 * I * H < 2^31; other shapes return MOE_ERR_UNSUPPORTED_SHAPE before anything
 * is enqueued.
 */
size_t moe_expert_ffn_workspace(moe_dims_t dims, int32_t T, moe_regime_t regime);
moe_status_t moe_expert_ffn(moe_dims_t dims, int32_t T, moe_regime_t regime,
                            const uint8_t* qx, const float* sx,
                            const int32_t* expert_offsets, const int32_t* sorted_src,
                            const uint8_t* w_gate, const float* s_gate,
                            const uint8_t* w_up, const float* s_up,
                            const uint8_t* w_down, const float* s_down,
                            float* y_rows, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * W8A16 expert FFN, decode regime (T <= MOE_DECODE_MAX_TOKENS): the paper's
 * own GEMV numerics (AVX-512 FP8 GEMV Kernel, post-scaling and scale-block
 * loop): bf16 activations, FP8 weights expanded to bf16, bf16 x bf16
 * products accumulated in fp32 over each 128-K block, the block's weight
 * scale applied once to the block sum, blocks summed in fp32:
 *   G[p,n] = sum_b s_gate_e[n/128,b] * (sum_{i in b} x[t,i] * W_gate_e[n,i])
 *   U likewise, h = bf16_rne(G * sigmoid(G) * U)   (bf16, the activation of down)
 *   y_rows[p,n] = sum_b s_down_e[n/128,b] * (sum_{i in b} h[p,i] * W_down_e[n,i])
 * No activation quantization: x_bf16 replaces qx/sx.  Other arguments as
 * in moe_expert_ffn (packed weight stacks, expert_offsets, sorted_src,
 * y_rows in expert-sorted order).  ws: moe_expert_ffn_w8a16_workspace(dims,
 * T) bytes, 256-byte aligned (bf16 h rows).  Errors as moe_expert_ffn;
 * T > MOE_DECODE_MAX_TOKENS is MOE_ERR_INVALID_ARG.
 */
size_t moe_expert_ffn_w8a16_workspace(moe_dims_t dims, int32_t T);
moe_status_t moe_expert_ffn_w8a16(moe_dims_t dims, int32_t T, const uint16_t* x_bf16,
                                  const int32_t* expert_offsets, const int32_t* sorted_src,
                                  const uint8_t* w_gate, const float* s_gate,
                                  const uint8_t* w_up, const float* s_up,
                                  const uint8_t* w_down, const float* s_down,
                                  float* y_rows, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Router-weighted combine (Operator Fusion for Quantized Inference: the
 * expert outputs are accumulated with the router weights in F32 and
 * converted back to the hidden type):
 *   out[t,n] = bf16_rne( sum_{j=0..k-1} topk_w[t,j] * y_rows[dest_row[t*k+j], n] )
 * summed in fp32 in slot order from +0.0.
 *
 * y_rows: device fp32 [T*k, H]; dest_row: device int32 [T*k];
 * topk_w: device fp32 [T, k]; out_bf16: device [T, H] bf16 bit patterns.
 */
moe_status_t moe_combine(const float* y_rows, const int32_t* dest_row, const float* topk_w,
                         int32_t T, int32_t k, int32_t H, uint16_t* out_bf16,
                         hipStream_t stream);

/*
 * Whole resident layer in one call: moe_quant_act -> moe_permute ->
 * moe_expert_ffn -> moe_combine on one stream, with the same arithmetic and
 * bit-identical results (the FP8 routed-expert FFN of System Design, run
 * from device memory), in fewer launches:
 *   T <= 256: quantization and the slot sort run as one launch;
 *   DECODE regime with T * k <= 16 and I <= 2048: the down projection and
 *   the combine run as one launch (a workgroup computes 16 output columns
 *   for every active expert and combines them per token in LDS);
 *   DECODE regime with T = 1, k <= 16, I <= 2048 and H <= 8192: two launches
 *   and no sort (one token's slots are distinct experts): the gate/up launch
 *   quantizes the token row itself and takes slot j's expert from topk_ids,
 *   writing h row j; the down + combine launch reads the same ids.
 * x_bf16: device [T, H] bf16 bits; topk_ids: device int32 [T, k];
 * topk_w: device fp32 [T, k]; weight stacks as in moe_expert_ffn (packed);
 * out_bf16: device [T, H] bf16 bits; dev_status: optional device int32
 * word, routing errors OR-ed in as by moe_permute (their outputs are
 * unspecified).  ws: moe_ffn_layer_workspace(dims, T, regime) bytes,
 * 256-byte aligned, owned by the caller; it holds the intermediate tensors
 * (qx, sx, expert offsets, sorted_src, dest_row, fp32 expert rows).  A
 * workspace must not be shared by calls that may overlap.  Argument errors
 * are returned before anything is enqueued (MOE_ERR_INVALID_ARG,
 * MOE_ERR_UNSUPPORTED_SHAPE, MOE_ERR_WORKSPACE); T == 0 does nothing.
 */
size_t moe_ffn_layer_workspace(moe_dims_t dims, int32_t T, moe_regime_t regime);
moe_status_t moe_ffn_layer(moe_dims_t dims, int32_t T, moe_regime_t regime, const uint16_t* x_bf16,
                           const int32_t* topk_ids, const float* topk_w,
                           const uint8_t* w_gate, const float* s_gate,
                           const uint8_t* w_up, const float* s_up,
                           const uint8_t* w_down, const float* s_down,
                           uint16_t* out_bf16, int32_t* dev_status,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_ffn_layer for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same call without the workspace arguments.  The layer's intermediate
 * tensors live in a device array of MOE_NOALLOC_SCRATCH_BYTES bytes inside
 * the library, one per GPU, held until the process ends; its device address
 * is looked up on the first call on each device.  The call allocates and
 * frees nothing and its results are bit-identical to moe_ffn_layer's.
 * A call whose moe_ffn_layer_workspace(dims, T, regime) exceeds
 * MOE_NOALLOC_SCRATCH_BYTES returns MOE_ERR_WORKSPACE before anything is
 * enqueued (DeepSeek-V3 shapes fit up to 64 decode tokens, or 128 prefill
 * tokens).  Other arguments, errors and T == 0 as in moe_ffn_layer.
 * All calls on one GPU share its scratch array, which keeps the last call's
 * contents (nothing in it needs clearing): calls that may overlap on one GPU
 * (different streams, or host threads without ordering) race.
 */
#define MOE_NOALLOC_SCRATCH_BYTES (32u << 20)
moe_status_t moe_ffn_layer_noalloc(moe_dims_t dims, int32_t T, moe_regime_t regime, const uint16_t* x_bf16,
                                   const int32_t* topk_ids, const float* topk_w,
                                   const uint8_t* w_gate, const float* s_gate,
                                   const uint8_t* w_up, const float* s_up,
                                   const uint8_t* w_down, const float* s_down,
                                   uint16_t* out_bf16, int32_t* dev_status, hipStream_t stream);

/*
 * Router (gate): the step before moe_permute.  The paper's Background on
 * Mixture-of-Experts names top-k and grouped top-k gating and SmallEP runs
 * the gate locally before sorting tokens; it fixes no formula, so the rule
 * is the DeepSeek-V3 gate:
 *   logits[t,e] = sum_i x[t,i] * W_r[e,i]    (bf16 inputs, fp32 accumulation)
 *   s = 1 / (1 + exp(-logits)),  key = s + bias[e]
 *   the E experts form n_group contiguous groups scored by the sum of their
 *   two largest keys; the topk_group best groups are kept; the k largest
 *   keys among their experts are chosen, listed by decreasing key;
 *   equal values go to the lower group / expert index;
 *   topk_w[t,j] = s[id_j] / (s[id_0] + ... + s[id_k-1]) * routed_scaling.
 * n_group = topk_group = 1 is plain top-k.
 *
 * x_bf16: device [T, H] bf16, 16-byte aligned; w_router_bf16: device [E, H]
 * bf16, 16-byte aligned; bias: device fp32 [E] or NULL (zero).
 * topk_ids: device int32 [T, k]; topk_w: device fp32 [T, k].  With
 * cfg.shared_expert >= 0 (the model's shared expert, always active, the
 * paper's Background on DeepSeek's shared experts) both are [T, k + 1] and
 * slot k holds (shared_expert, 1.0): with that expert's weights at index
 * shared_expert of the stacks (E + 1 experts in moe_permute and
 * moe_expert_ffn) the rest of the path adds it after the routed experts,
 * out = bf16(sum_j w_j y_j + y_shared), with no other change.
 * ws: device, moe_router_workspace(T, H, E) bytes (partial logits).
 * Requires H % 32 == 0, 1 <= E <= 1024, n_group <= 64 dividing E with at
 * least two experts per group when n_group > 1, 1 <= topk_group <= n_group,
 * 1 <= k <= min(32, topk_group * E / n_group) (k <= 31 with a shared
 * expert), routed_scaling > 0; else
 * MOE_ERR_INVALID_ARG before any launch.  Inputs must be finite.
 */
typedef struct {
  int32_t n_group;       /* expert groups (1: no group limit) */
  int32_t topk_group;    /* groups kept per token */
  float routed_scaling;  /* factor on the normalised weights */
  int32_t shared_expert; /* < 0: none; else this id is appended as slot k with weight 1.0 */
} moe_router_cfg_t;
size_t moe_router_workspace(int32_t T, int32_t H, int32_t E);
moe_status_t moe_router(const uint16_t* x_bf16, int32_t T, int32_t H, const uint16_t* w_router_bf16,
                        const float* bias, int32_t E, int32_t k, moe_router_cfg_t cfg,
                        int32_t* topk_ids, float* topk_w, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/*
 * Stream-loaded layer (System Design, Stream-loading Prefill: a loader
 * stages each expert's weights from host memory into a device experts ring
 * buffer and sets an ON event, the model waits for ON, runs the expert and
 * sets an OFF event, and the slot is reused without copying back).
 *
 * The whole layer (quantize, permute, expert FFN, combine) with the expert
 * weights in pinned host memory.  Expert e is copied on `copy` into ring
 * slot e % ring_slots (waiting for that slot's previous expert to finish),
 * then run on `compute` over every chunk's rows of e as soon as its copy
 * lands.  Tokens are permuted and combined per chunk of chunk_tokens.  Each
 * output row equals moe_expert_ffn with MOE_REGIME_PREFILL on resident
 * weights bit for bit (same kernels, same per-row arithmetic).
 *
 * host_w_*: pinned host e4m3 weights, packed as for moe_expert_ffn ([E,I,H]
 * for gate/up, [E,H,I] for down, each expert's matrix in the layout of
 * moe_pack_weight; row-major stacks give undefined results); host_s_*:
 * pinned host fp32 scales.
 * dev_ring: device, moe_ring_bytes(dims, slots) bytes, three sub-rings
 * [slots][I*H] of W_gate, W_up and [slots][H*I] of W_down (slot s holds one
 * expert in each).  dev_ring_scales: device, moe_ring_scale_bytes(dims,
 * slots) bytes, the same three sub-rings of scales.  Experts are copied and
 * run in groups of consecutive experts (a divisor of the slot count) so
 * that each launch fills the GPU.  ctx: from moe_stream_ctx_create
 * with the same slot count.  Its per-slot events order the ring across
 * calls: calls on one ctx (the layers of a model streamed through one ring)
 * may be enqueued back to back without a host synchronisation; a slot is
 * refilled only after the kernels of earlier calls that read it have run,
 * and the next call's copies start as soon as slots free up.  A ctx must not
 * be used by two host threads at once.  x_bf16, topk_ids, topk_w, out_bf16 as in the other calls (device).
 * ws: device, moe_ffn_streamed_workspace(dims, T, chunk_tokens) bytes, 256-byte
 * aligned (it holds the fp32 expert rows of all T*k slots).  compute and copy
 * should be distinct streams for the copies to overlap the kernels.
 * Shapes: the PREFILL limits of moe_expert_ffn (H % 256 == 0,
 * max(H, I) <= 24576, I * H < 2^31); others return
 * MOE_ERR_UNSUPPORTED_SHAPE before anything is enqueued.
 */
typedef struct moe_stream_ctx* moe_stream_ctx_t;
moe_status_t moe_stream_ctx_create(int32_t ring_slots, moe_stream_ctx_t* out);
void moe_stream_ctx_destroy(moe_stream_ctx_t ctx);
size_t moe_ring_bytes(moe_dims_t dims, int32_t ring_slots);
size_t moe_ring_scale_bytes(moe_dims_t dims, int32_t ring_slots);
size_t moe_ffn_streamed_workspace(moe_dims_t dims, int32_t T, int32_t chunk_tokens);
moe_status_t moe_ffn_streamed(moe_dims_t dims, int32_t T, int32_t chunk_tokens, const uint16_t* x_bf16,
                              const int32_t* topk_ids, const float* topk_w,
                              const uint8_t* host_w_gate, const float* host_s_gate,
                              const uint8_t* host_w_up, const float* host_s_up,
                              const uint8_t* host_w_down, const float* host_s_down,
                              uint8_t* dev_ring, float* dev_ring_scales, moe_stream_ctx_t ctx,
                              uint16_t* out_bf16, int32_t* dev_status, void* ws, size_t ws_bytes,
                              hipStream_t compute, hipStream_t copy);

/*
 * The ring schedule that moe_ffn_streamed enqueues for one layer (System
 * Design, Stream-loading Prefill: the loader's copies with their ON events,
 * the model's launches with their OFF events), computed on the host without
 * any GPU call, for testing and inspection.  Experts go in groups of
 * consecutive experts in slots expert mod ring_slots; per group, in enqueue
 * order: on the copy stream WAIT_OFF(s) for each slot s of the group that
 * already holds an OFF record, COPY, RECORD_ON(first slot); on the compute
 * stream WAIT_ON(first slot), LAUNCH, RECORD_OFF(s) for each slot.  A wait
 * refers to the latest record of that event enqueued before it.
 *
 * op fields: WAIT_OFF, RECORD_ON, WAIT_ON, RECORD_OFF: a = slot;
 * COPY: experts a .. a + b - 1 into slots c .. c + b - 1; LAUNCH: the FFN of
 * experts a .. a + b - 1 read from slots c .. c + b - 1.
 * off_recorded: host uint8[ring_slots], nonzero where a slot holds an OFF
 * record from an earlier call on the same ring (zeros for a new context);
 * updated in place, as a call leaves the context.  ops: host array of cap
 * entries; *n_ops receives the count.  Returns MOE_ERR_WORKSPACE (with
 * *n_ops set, ops and off_recorded untouched) when cap is too small, and the
 * argument and shape errors of moe_ffn_streamed.  T == 0 gives no ops.
 */
typedef struct {
  int32_t op;       /* MOE_SOP_* */
  int32_t a, b, c;
} moe_stream_op_t;
#define MOE_SOP_WAIT_OFF 1
#define MOE_SOP_COPY 2
#define MOE_SOP_RECORD_ON 3
#define MOE_SOP_WAIT_ON 4
#define MOE_SOP_LAUNCH 5
#define MOE_SOP_RECORD_OFF 6
moe_status_t moe_stream_schedule(moe_dims_t dims, int32_t T, int32_t chunk_tokens, int32_t ring_slots,
                                 uint8_t* off_recorded, moe_stream_op_t* ops, int32_t cap, int32_t* n_ops);

/*
 * Diagnostics: per-launch kernel timing.  After moe_profile_begin(n), every
 * kernel launch of the library (at most n) is bracketed by two HIP events
 * recorded on its stream.  moe_profile_end() stops recording, waits for the
 * recorded events and returns the number of launches; moe_profile_get(i)
 * gives launch i's kernel name (static storage) and duration in ms.  The
 * events are created by the library on the first begin and kept; use from
 * one host thread at a time.
 */
moe_status_t moe_profile_begin(int32_t max_launches);
int32_t moe_profile_end(void);
moe_status_t moe_profile_get(int32_t i, float* ms, const char** name);

#ifdef __cplusplus
}
#endif

#endif /* MOE_FP8_MI355X_H */
