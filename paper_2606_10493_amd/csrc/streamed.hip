// Stream-loading of one routed-expert layer whose FP8 weights stay in pinned
// host memory (the paper's stream-loading prefill, System Design: a loader
// stages each expert's weights into an experts ring buffer on the device and
// signals an ON event; the model runs the expert after waiting for it and
// signals an OFF event; the slot is then reused without copying anything
// back, the host copy being authoritative).
//
// MI355X form: one host thread enqueues everything.  The loader is a copy
// stream issuing hipMemcpyAsync from pinned host memory into the ring; the
// model is the caller's compute stream; ON/OFF are HIP events per group of
// slots (stream-ordered, so the paper's host-side threading events are not
// needed).  Experts go in groups of G consecutive experts held in G
// consecutive slots (the ring is three sub-rings, gate | up | down, each
// [R][matrix], so a group looks like a small weight tensor to the kernels).
// G is the largest divisor of R, at most R / 2, that gives about 2048 rows
// per launch, so a launch fills the GPU and the ring has two slot groups or
// more.  Enqueue order per group g (slot group v = g mod R/G):
//   copy:    [wait OFF[v] if g >= R/G]  6 copies (W, S of gate/up/down)  record ON[v]
//   compute: wait ON[v]  FFN(group) over every chunk's rows           record OFF[v]
// Because copy(g) is enqueued after compute(g - R/G) and compute(g) after
// copy(g), every wait refers to the intended record.
//
// Tokens: all T are quantized at once; the permutation and the combine work
// per chunk of chunk_tokens tokens.  The FFN of a group is one launch pair
// (gate/up, down) over its rows in every chunk, read through a G-expert
// window of each chunk's offsets (offsets pointer + e0): an expert's rows of
// all chunks are numbered as one run of launch rows (tables map each to its
// sorted position and token), so its 128-row tiles span chunks and read its
// weight slices together.  The kernels and every row's arithmetic are those
// of the resident path: each output row is bit-identical to moe_expert_ffn
// with the prefill regime.
#include <vector>

#include "common.h"

struct moe_stream_ctx {
  int32_t slots;
  std::vector<hipEvent_t> on, off;  // per ring slot
  std::vector<char> off_recorded;   // off[s] holds the last kernels that read slot s (this call or an earlier one)
};

namespace moe {

moe_status_t run_ffn_prefill_view(const moe_dims_t& d, const PrefillRows& r, const uint8_t* qx, const float* sx,
                                  const int32_t* sorted_src, const uint8_t* w_gate, const float* s_gate,
                                  const uint8_t* w_up, const float* s_up, const uint8_t* w_down, const float* s_down,
                                  float* y_rows, uint8_t* qh, float* sh, int32_t* tiles, hipStream_t stream);
size_t prefill_tiles_bytes(int64_t n_units, int64_t max_mtiles, int64_t table_rows);
moe_status_t prefill_shape_check(const moe_dims_t& d);

namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct StreamLayout {
  size_t qx, sx, offsets, sorted_src, dest_row, perm_ws, qh, sh, tiles, y, total;
  int64_t n_chunks, chunk;
};

StreamLayout layout(const moe_dims_t& d, int32_t T, int32_t chunk_tokens) {
  StreamLayout L{};
  const int64_t H = d.hidden, I = d.inter, E = d.n_experts, k = d.topk;
  L.chunk = chunk_tokens;
  L.n_chunks = ((int64_t)T + chunk_tokens - 1) / chunk_tokens;
  const int64_t ck = (int64_t)chunk_tokens * k;  // rows of one chunk
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  L.qx = take((size_t)T * H);
  L.sx = take((size_t)T * (H / kBlock) * sizeof(float));
  L.offsets = take((size_t)L.n_chunks * (E + 1) * sizeof(int32_t));
  L.sorted_src = take((size_t)L.n_chunks * ck * sizeof(int32_t));
  L.dest_row = take((size_t)L.n_chunks * ck * sizeof(int32_t));
  L.perm_ws = take(moe_permute_workspace(chunk_tokens, d.topk, d.n_experts));
  const int64_t R = (int64_t)T * k;  // sorted rows of all chunks
  L.qh = take((size_t)R * I);
  L.sh = take((size_t)R * (I / kBlock) * sizeof(float));
  // G <= E experts over all chunks (row tables of all rows)
  L.tiles = take(prefill_tiles_bytes(E, (R + 127) / 128 + E, R));
  L.y = take((size_t)R * H * sizeof(float));
  L.total = off;
  return L;
}

// Experts per slot group: the largest divisor of R, at most R / 2 when R > 1
// (so the ring has two slot groups or more and a group's copy overlaps the
// previous group's kernels: a ping-pong ring at R = 2), that gives about
// 2048 rows per chunk to a launch.
int ring_group_size(int64_t chunk_tokens, int64_t k, int64_t E, int R) {
  const int64_t rows_per_expert = (chunk_tokens * k + E - 1) / E;
  int64_t want = (2048 + rows_per_expert - 1) / rows_per_expert;
  const int64_t cap = R > 1 ? R / 2 : 1;
  if (want > cap) want = cap;
  for (int g = (int)want; g >= 1; --g)
    if (R % g == 0) return g;
  return 1;
}

// The ring schedule of one layer call in enqueue order (host only).  Per
// group of G consecutive experts e0 .. e0 + g - 1 in slots slot0 = e0 mod R
// onwards:
//   copy stream:    WAIT_OFF(s) for each slot s of the group that holds an
//                   OFF record (the kernels that read it last, in this call
//                   or an earlier one), COPY(e0, g, slot0), RECORD_ON(slot0);
//   compute stream: WAIT_ON(slot0), LAUNCH(e0, g, slot0), RECORD_OFF(s) for
//                   each slot of the group.
// A wait refers to the event's latest record enqueued before it, so copy(g)
// (enqueued after compute(g - R/G)) waits for that compute, and compute(g)
// for copy(g).  off_recorded (one flag per slot, in/out) carries the OFF
// records across calls on one ring.
void plan_ring(int64_t E, int G, int R, std::vector<char>& off_recorded, std::vector<moe_stream_op_t>& ops) {
  for (int64_t e0 = 0; e0 < E; e0 += G) {
    const int g = (int)((E - e0) < G ? (E - e0) : G);
    const int slot0 = (int)(e0 % R);
    for (int s = slot0; s < slot0 + g; ++s)
      if (off_recorded[s]) ops.push_back({MOE_SOP_WAIT_OFF, s, 0, 0});
    ops.push_back({MOE_SOP_COPY, (int32_t)e0, g, slot0});
    ops.push_back({MOE_SOP_RECORD_ON, slot0, 0, 0});
    ops.push_back({MOE_SOP_WAIT_ON, slot0, 0, 0});
    ops.push_back({MOE_SOP_LAUNCH, (int32_t)e0, g, slot0});
    for (int s = slot0; s < slot0 + g; ++s) {
      ops.push_back({MOE_SOP_RECORD_OFF, s, 0, 0});
      off_recorded[s] = 1;
    }
  }
}

moe_status_t check_streamed_dims(const moe_dims_t& d, int32_t T, int32_t chunk_tokens, const char* who) {
  if (d.hidden <= 0 || d.inter <= 0 || d.n_experts < 1 || d.n_experts > 1024 || d.topk < 1 || d.topk > 32 ||
      d.topk > d.n_experts || T < 0 || chunk_tokens < 1)
    return fail(MOE_ERR_INVALID_ARG, "%s: H=%d I=%d E=%d k=%d T=%d chunk=%d", who, d.hidden, d.inter, d.n_experts,
                d.topk, T, chunk_tokens);
  if (d.hidden % 256 || d.inter % kBlock)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "%s: H must be a multiple of 256 and I of 128", who);
  // The prefill kernels' limits (K, LDS, expert matrix size), before anything is enqueued.
  return prefill_shape_check(d);
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" size_t moe_ring_bytes(moe_dims_t d, int32_t slots) {
  if (slots < 1 || d.hidden <= 0 || d.inter <= 0) return 0;
  return (size_t)slots * 3 * (size_t)d.hidden * d.inter;
}

extern "C" size_t moe_ring_scale_bytes(moe_dims_t d, int32_t slots) {
  if (slots < 1 || d.hidden <= 0 || d.inter <= 0) return 0;
  return (size_t)slots * 3 * (size_t)(d.hidden / kBlock) * (d.inter / kBlock) * sizeof(float);
}

extern "C" moe_status_t moe_stream_ctx_create(int32_t ring_slots, moe_stream_ctx_t* out) {
  if (!out || ring_slots < 1 || ring_slots > 4096)
    return fail(MOE_ERR_INVALID_ARG, "moe_stream_ctx_create: ring_slots=%d", ring_slots);
  *out = nullptr;
  moe_stream_ctx* c = new moe_stream_ctx;
  c->slots = ring_slots;
  c->on.resize(ring_slots);
  c->off.resize(ring_slots);
  c->off_recorded.assign(ring_slots, 0);
  for (int i = 0; i < ring_slots; ++i) {
    if (hipEventCreateWithFlags(&c->on[i], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&c->off[i], hipEventDisableTiming) != hipSuccess) {
      for (int j = 0; j <= i; ++j) {
        if (c->on[j]) (void)hipEventDestroy(c->on[j]);
        if (c->off[j]) (void)hipEventDestroy(c->off[j]);
      }
      delete c;
      return fail(MOE_ERR_HIP, "moe_stream_ctx_create: hipEventCreate failed");
    }
  }
  *out = c;
  return MOE_OK;
}

extern "C" void moe_stream_ctx_destroy(moe_stream_ctx_t ctx) {
  if (!ctx) return;
  for (auto e : ctx->on) (void)hipEventDestroy(e);
  for (auto e : ctx->off) (void)hipEventDestroy(e);
  delete ctx;
}

extern "C" size_t moe_ffn_streamed_workspace(moe_dims_t d, int32_t T, int32_t chunk_tokens) {
  if (T < 0 || chunk_tokens < 1 || d.hidden <= 0 || d.inter <= 0 || d.n_experts <= 0 || d.topk <= 0) return 0;
  return layout(d, T, chunk_tokens).total;
}

extern "C" moe_status_t moe_stream_schedule(moe_dims_t d, int32_t T, int32_t chunk_tokens, int32_t ring_slots,
                                            uint8_t* off_recorded, moe_stream_op_t* ops, int32_t cap,
                                            int32_t* n_ops) {
  moe_status_t st = check_streamed_dims(d, T, chunk_tokens, "moe_stream_schedule");
  if (st != MOE_OK) return st;
  if (ring_slots < 1 || ring_slots > 4096 || !off_recorded || !n_ops || cap < 0)
    return fail(MOE_ERR_INVALID_ARG, "moe_stream_schedule: ring_slots=%d cap=%d", ring_slots, cap);
  *n_ops = 0;
  if (T == 0) return MOE_OK;
  std::vector<char> rec(ring_slots);
  for (int s = 0; s < ring_slots; ++s) rec[s] = off_recorded[s] ? 1 : 0;
  std::vector<moe_stream_op_t> plan;
  plan_ring(d.n_experts, ring_group_size(chunk_tokens, d.topk, d.n_experts, ring_slots), ring_slots, rec, plan);
  *n_ops = (int32_t)plan.size();
  if (!ops || cap < (int32_t)plan.size())
    return fail(MOE_ERR_WORKSPACE, "moe_stream_schedule: %d ops, room for %d", (int)plan.size(), cap);
  for (size_t i = 0; i < plan.size(); ++i) ops[i] = plan[i];
  for (int s = 0; s < ring_slots; ++s) off_recorded[s] = (uint8_t)rec[s];
  return MOE_OK;
}

extern "C" moe_status_t moe_ffn_streamed(moe_dims_t d, int32_t T, int32_t chunk_tokens, const uint16_t* x_bf16,
                                         const int32_t* topk_ids, const float* topk_w, const uint8_t* host_w_gate,
                                         const float* host_s_gate, const uint8_t* host_w_up, const float* host_s_up,
                                         const uint8_t* host_w_down, const float* host_s_down, uint8_t* dev_ring,
                                         float* dev_ring_scales, moe_stream_ctx_t ctx, uint16_t* out_bf16,
                                         int32_t* dev_status, void* ws, size_t ws_bytes, hipStream_t compute,
                                         hipStream_t copy) {
  moe_status_t st0 = check_streamed_dims(d, T, chunk_tokens, "moe_ffn_streamed");
  if (st0 != MOE_OK) return st0;
  if (!ctx) return fail(MOE_ERR_INVALID_ARG, "moe_ffn_streamed: null stream context");
  if (T == 0) return MOE_OK;
  if ((int64_t)T * d.topk > 0x7fffffff) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_ffn_streamed: T*k overflows");
  if (!x_bf16 || !topk_ids || !topk_w || !host_w_gate || !host_s_gate || !host_w_up || !host_s_up || !host_w_down ||
      !host_s_down || !dev_ring || !dev_ring_scales || !out_bf16)
    return fail(MOE_ERR_INVALID_ARG, "moe_ffn_streamed: null pointer");
  if (!aligned(dev_ring, 16) || !aligned(x_bf16, 16) || !aligned(out_bf16, 16) || !aligned(ws, 256))
    return fail(MOE_ERR_INVALID_ARG, "moe_ffn_streamed: misaligned pointer");
  const StreamLayout L = layout(d, T, chunk_tokens);
  if (!ws || ws_bytes < L.total)
    return fail(MOE_ERR_WORKSPACE, "moe_ffn_streamed: workspace %zu bytes < %zu", ws_bytes, L.total);

  uint8_t* base = static_cast<uint8_t*>(ws);
  uint8_t* qx = base + L.qx;
  float* sx = reinterpret_cast<float*>(base + L.sx);
  int32_t* offsets = reinterpret_cast<int32_t*>(base + L.offsets);
  int32_t* sorted_src = reinterpret_cast<int32_t*>(base + L.sorted_src);
  int32_t* dest_row = reinterpret_cast<int32_t*>(base + L.dest_row);
  void* perm_ws = base + L.perm_ws;
  uint8_t* qh = base + L.qh;
  float* sh = reinterpret_cast<float*>(base + L.sh);
  int32_t* tiles = reinterpret_cast<int32_t*>(base + L.tiles);
  float* y = reinterpret_cast<float*>(base + L.y);

  const int64_t H = d.hidden, I = d.inter, E = d.n_experts, k = d.topk;
  const size_t wmat = (size_t)I * H;                                   // bytes of one expert matrix
  const size_t smat = (size_t)(I / kBlock) * (H / kBlock);             // scales of one expert matrix
  const int R = ctx->slots;

  // Quantize every token, then permute each chunk (compute stream).
  moe_status_t st = moe_quant_act(x_bf16, T, d.hidden, qx, sx, compute);
  if (st != MOE_OK) return st;
  const size_t perm_ws_bytes = moe_permute_workspace(chunk_tokens, d.topk, d.n_experts);
  for (int64_t c = 0; c < L.n_chunks; ++c) {
    const int32_t t0 = (int32_t)(c * L.chunk);
    const int32_t tc = (int32_t)((T - t0) < L.chunk ? (T - t0) : L.chunk);
    st = moe_permute(topk_ids + (int64_t)t0 * k, tc, d.topk, d.n_experts, offsets + c * (E + 1),
                     sorted_src + c * L.chunk * k, dest_row + c * L.chunk * k, dev_status, perm_ws, perm_ws_bytes,
                     compute);
    if (st != MOE_OK) return st;
  }

  // Experts are streamed and run in groups of G consecutive experts, held in
  // G consecutive ring slots; one GEMM launch pair covers the group's rows
  // of every chunk (an expert's tiles span chunks).  The schedule
  // (plan_ring) is executed op by op.
  const int G = ring_group_size(L.chunk, k, E, R);
  std::vector<moe_stream_op_t> plan;
  {
    std::vector<char> rec(ctx->off_recorded);
    plan_ring(E, G, R, rec, plan);
  }
  uint8_t* ring_gate = dev_ring;
  uint8_t* ring_up = dev_ring + (size_t)R * wmat;
  uint8_t* ring_down = dev_ring + 2 * (size_t)R * wmat;
  float* ring_sgate = dev_ring_scales;
  float* ring_sup = dev_ring_scales + (size_t)R * smat;
  float* ring_sdown = dev_ring_scales + 2 * (size_t)R * smat;
  for (const moe_stream_op_t& op : plan) {
    switch (op.op) {
      case MOE_SOP_WAIT_OFF:  // loader: the slot is free once the kernels that read it last ran
        if (hipStreamWaitEvent(copy, ctx->off[op.a], 0) != hipSuccess)
          return fail(MOE_ERR_HIP, "moe_ffn_streamed: wait OFF");
        break;
      case MOE_SOP_COPY: {
        const int64_t e0 = op.a;
        const int slot0 = op.c;
        const size_t nb_w = (size_t)op.b * wmat, nb_s = (size_t)op.b * smat * sizeof(float);
        if (hipMemcpyAsync(ring_gate + slot0 * wmat, host_w_gate + e0 * wmat, nb_w, hipMemcpyHostToDevice, copy) ||
            hipMemcpyAsync(ring_up + slot0 * wmat, host_w_up + e0 * wmat, nb_w, hipMemcpyHostToDevice, copy) ||
            hipMemcpyAsync(ring_down + slot0 * wmat, host_w_down + e0 * wmat, nb_w, hipMemcpyHostToDevice, copy) ||
            hipMemcpyAsync(ring_sgate + slot0 * smat, host_s_gate + e0 * smat, nb_s, hipMemcpyHostToDevice, copy) ||
            hipMemcpyAsync(ring_sup + slot0 * smat, host_s_up + e0 * smat, nb_s, hipMemcpyHostToDevice, copy) ||
            hipMemcpyAsync(ring_sdown + slot0 * smat, host_s_down + e0 * smat, nb_s, hipMemcpyHostToDevice, copy))
          return fail(MOE_ERR_HIP, "moe_ffn_streamed: copy of experts %lld..", (long long)e0);
        break;
      }
      case MOE_SOP_RECORD_ON:
        if (hipEventRecord(ctx->on[op.a], copy) != hipSuccess) return fail(MOE_ERR_HIP, "moe_ffn_streamed: record ON");
        break;
      case MOE_SOP_WAIT_ON:
        if (hipStreamWaitEvent(compute, ctx->on[op.a], 0) != hipSuccess)
          return fail(MOE_ERR_HIP, "moe_ffn_streamed: wait ON");
        break;
      case MOE_SOP_LAUNCH: {  // model: the group's rows of every chunk in one launch pair
        const int64_t e0 = op.a;
        const int g_here = op.b, slot0 = op.c;
        PrefillRows rows{};
        rows.offsets = offsets + e0;
        rows.off_stride = E + 1;
        rows.n_units = g_here;
        rows.n_chunks = (int)L.n_chunks;
        rows.chunk_rows = L.chunk * k;
        rows.chunk_tokens = (int)L.chunk;
        rows.tokens = T;
        rows.rows = (int64_t)T * k;
        rows.max_mtiles = (rows.rows + 127) / 128 + g_here;
        const moe_dims_t vd{d.hidden, d.inter, g_here, d.topk};
        st = run_ffn_prefill_view(vd, rows, qx, sx, sorted_src, ring_gate + slot0 * wmat, ring_sgate + slot0 * smat,
                                  ring_up + slot0 * wmat, ring_sup + slot0 * smat, ring_down + slot0 * wmat,
                                  ring_sdown + slot0 * smat, y, qh, sh, tiles, compute);
        if (st != MOE_OK) return st;
        break;
      }
      case MOE_SOP_RECORD_OFF:
        if (hipEventRecord(ctx->off[op.a], compute) != hipSuccess)
          return fail(MOE_ERR_HIP, "moe_ffn_streamed: record OFF");
        ctx->off_recorded[op.a] = 1;
        break;
      default:
        return fail(MOE_ERR_INVALID_ARG, "moe_ffn_streamed: bad schedule op %d", op.op);
    }
  }

  // Combine each chunk.
  for (int64_t c = 0; c < L.n_chunks; ++c) {
    const int32_t t0 = (int32_t)(c * L.chunk);
    const int32_t tc = (int32_t)((T - t0) < L.chunk ? (T - t0) : L.chunk);
    st = moe_combine(y + c * L.chunk * k * H, dest_row + c * L.chunk * k, topk_w + (int64_t)t0 * k, tc, d.topk,
                     d.hidden, out_bf16 + (int64_t)t0 * H, compute);
    if (st != MOE_OK) return st;
  }
  return MOE_OK;
}
