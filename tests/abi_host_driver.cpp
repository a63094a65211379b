// Host-side paths of the C ABI, for a build with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code (tests/test_abi_sanitizers.py
// builds the library sources with the device code left out and links this
// file).  Every call here returns before anything is enqueued: argument and
// shape errors, workspace-size queries over extreme sizes, the streamed
// layer's ring schedule, the status strings.  Nothing touches a GPU.
//
// Exits 0 when every call returned the expected status; a sanitizer report
// (out-of-bounds access, signed overflow, misaligned or null access in host
// code) is the other failure this build looks for.
#include <climits>
#include <cstdio>
#include <cstring>
#include <vector>

#include "moe.h"

namespace {

int g_failures = 0;
int g_calls = 0;

void expect(moe_status_t got, moe_status_t want, const char* what, int line) {
  ++g_calls;
  if (got != want) {
    ++g_failures;
    std::printf("line %d: %s returned %d (%s), expected %d; last error: %s\n", line, what, (int)got,
                moe_status_string(got), (int)want, moe_last_error());
  }
}

void expect_not_ok(moe_status_t got, const char* what, int line) {
  ++g_calls;
  if (got == MOE_OK) {
    ++g_failures;
    std::printf("line %d: %s returned MOE_OK on invalid arguments\n", line, what);
  }
}

#define EXPECT(call, want) expect((call), (want), #call, __LINE__)
#define EXPECT_ERR(call) expect_not_ok((call), #call, __LINE__)

// Stand-ins for device pointers: never dereferenced on these paths.
template <typename T>
T* fake(uintptr_t at) {
  return reinterpret_cast<T*>(at);
}

const int32_t kTs[] = {-1, 0, 1, 2, 16, 63, 64, 65, 255, 256, 257, 4096, 65536, 1 << 20, INT32_MAX};
const moe_dims_t kDims[] = {
    {256, 128, 8, 2},     {7168, 2048, 256, 8}, {24576, 24576, 1024, 32}, {7168, 2048, 1, 1},
    {0, 128, 8, 2},       {256, 0, 8, 2},       {384, 128, 8, 2},         {200, 128, 8, 2},
    {256, 100, 8, 2},     {256, 128, 0, 1},     {256, 128, 8, 9},         {256, 128, 8, 0},
    {256, 128, 2048, 8},  {INT32_MAX, 128, 8, 2}, {256, INT32_MAX, 8, 2}, {-256, -128, -8, -2},
};
const moe_regime_t kRegimes[] = {MOE_REGIME_AUTO, MOE_REGIME_DECODE, MOE_REGIME_PREFILL, (moe_regime_t)7};

void workspace_queries() {
  size_t sink = 0;
  for (int32_t T : kTs) {
    for (int32_t k : {-1, 0, 1, 8, 32, 33})
      for (int32_t E : {-1, 0, 1, 8, 256, 1024, 1025}) sink ^= moe_permute_workspace(T, k, E);
    for (const moe_dims_t& d : kDims) {
      for (moe_regime_t rg : kRegimes) {
        sink ^= moe_expert_ffn_workspace(d, T, rg);
        sink ^= moe_ffn_layer_workspace(d, T, rg);
      }
      sink ^= moe_expert_ffn_w8a16_workspace(d, T);
      for (int32_t chunk : {-1, 0, 1, 256, 4096, INT32_MAX}) sink ^= moe_ffn_streamed_workspace(d, T, chunk);
    }
    for (int32_t H : {-1, 0, 32, 7168, INT32_MAX})
      for (int32_t E : {-1, 0, 1, 256, 1024, 1025}) sink ^= moe_router_workspace(T, H, E);
  }
  for (const moe_dims_t& d : kDims)
    for (int32_t R : {-1, 0, 1, 2, 256, 4096, INT32_MAX}) {
      sink ^= moe_ring_bytes(d, R);
      sink ^= moe_ring_scale_bytes(d, R);
    }
  std::printf("workspace queries done (%zx)\n", sink & 0xf);
}

void ring_schedules() {
  int n_schedules = 0;
  for (int32_t R : {1, 2, 3, 5, 16, 32, 256, 4096}) {
    for (int32_t E : {1, 7, 256, 1024}) {
      std::vector<uint8_t> rec(R, 0);
      for (int32_t T : {0, 1, 300, 32768}) {
        for (int32_t chunk : {1, 256, 4096, 65536}) {
          const moe_dims_t d{256, 128, E, E < 8 ? 1 : 8};
          int32_t n = -1;
          EXPECT(moe_stream_schedule(d, T, chunk, R, rec.data(), nullptr, 0, &n),
                 T == 0 ? MOE_OK : MOE_ERR_WORKSPACE);
          std::vector<moe_stream_op_t> ops(n > 0 ? n : 1);
          int32_t n2 = -1;
          EXPECT(moe_stream_schedule(d, T, chunk, R, rec.data(), ops.data(), n, &n2), MOE_OK);
          if (n2 != n) {
            ++g_failures;
            std::printf("schedule size changed: %d then %d\n", n, n2);
          }
          ++n_schedules;
        }
      }
    }
  }
  const moe_dims_t d{256, 128, 8, 2};
  std::vector<uint8_t> rec(4, 0);
  int32_t n = 0;
  EXPECT(moe_stream_schedule(d, 16, 16, 0, rec.data(), nullptr, 0, &n), MOE_ERR_INVALID_ARG);
  EXPECT(moe_stream_schedule(d, 16, 16, 4, nullptr, nullptr, 0, &n), MOE_ERR_INVALID_ARG);
  EXPECT(moe_stream_schedule(d, 16, 16, 4, rec.data(), nullptr, 0, nullptr), MOE_ERR_INVALID_ARG);
  EXPECT(moe_stream_schedule(d, 16, 16, 4, rec.data(), nullptr, -1, &n), MOE_ERR_INVALID_ARG);
  EXPECT(moe_stream_schedule(d, 16, 0, 4, rec.data(), nullptr, 0, &n), MOE_ERR_INVALID_ARG);
  EXPECT(moe_stream_schedule(moe_dims_t{384, 128, 8, 2}, 16, 16, 4, rec.data(), nullptr, 0, &n),
         MOE_ERR_UNSUPPORTED_SHAPE);
  std::printf("ring schedules done (%d)\n", n_schedules);
}

void argument_errors() {
  const uint16_t* x = fake<const uint16_t>(0x10000);
  const float* f = fake<const float>(0x20000);
  const uint8_t* q = fake<const uint8_t>(0x30000);
  const int32_t* ids = fake<const int32_t>(0x40000);
  uint8_t* qo = fake<uint8_t>(0x50000);
  float* fo = fake<float>(0x60000);
  int32_t* io = fake<int32_t>(0x70000);
  uint16_t* xo = fake<uint16_t>(0x80000);
  const moe_dims_t ds{7168, 2048, 256, 8};

  // quantizers and packing
  EXPECT_ERR(moe_quant_act(nullptr, 4, 256, qo, fo, nullptr));
  EXPECT_ERR(moe_quant_act(x, -1, 256, qo, fo, nullptr));
  EXPECT_ERR(moe_quant_act(x, 4, 200, qo, fo, nullptr));
  EXPECT_ERR(moe_quant_act(x, 4, 0, qo, fo, nullptr));
  EXPECT_ERR(moe_quant_act(x, INT32_MAX, INT32_MAX - 127, qo, fo, nullptr));
  EXPECT_ERR(moe_quant_rows_f32(f, 4, 256, nullptr, fo, nullptr));
  EXPECT_ERR(moe_quant_rows_f32(f, 4, 100, qo, fo, nullptr));
  EXPECT_ERR(moe_quant_weight(f, 1, 100, 128, qo, fo, nullptr));
  EXPECT_ERR(moe_quant_weight(f, -1, 128, 128, qo, fo, nullptr));
  EXPECT_ERR(moe_quant_weight(nullptr, 1, 128, 128, qo, fo, nullptr));
  EXPECT_ERR(moe_pack_weight(q, 1, 100, 128, qo, nullptr));
  EXPECT_ERR(moe_pack_weight(q, 1, 128, 128, nullptr, nullptr));
  EXPECT_ERR(moe_pack_weight(q, INT32_MAX, 24576, 24576, qo, nullptr));

  // permutation
  EXPECT_ERR(moe_permute(nullptr, 4, 8, 256, io, io, io, nullptr, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_permute(ids, -1, 8, 256, io, io, io, nullptr, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_permute(ids, 4, 0, 256, io, io, io, nullptr, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_permute(ids, 4, 9, 8, io, io, io, nullptr, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_permute(ids, 4, 8, 2048, io, io, io, nullptr, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_permute(ids, INT32_MAX, 32, 256, io, io, io, nullptr, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_permute(ids, 100000, 8, 256, io, io, io, nullptr, nullptr, 0, nullptr));

  // expert FFN
  for (const moe_dims_t& d : kDims)
    for (moe_regime_t rg : kRegimes)
      for (int32_t T : {-1, 65, 4096}) {
        const moe_status_t st =
            moe_expert_ffn(d, T, rg, q, f, ids, ids, q, f, q, f, q, f, fo, nullptr, 0, nullptr);
        EXPECT_ERR(st);
      }
  EXPECT(moe_expert_ffn(ds, 0, MOE_REGIME_AUTO, q, f, ids, ids, q, f, q, f, q, f, fo, nullptr, 0, nullptr), MOE_OK);
  EXPECT_ERR(moe_expert_ffn(ds, 4, MOE_REGIME_AUTO, nullptr, f, ids, ids, q, f, q, f, q, f, fo, qo, 1 << 30,
                            nullptr));
  EXPECT_ERR(moe_expert_ffn(ds, 4, MOE_REGIME_AUTO, q, f, ids, ids, q + 1, f, q, f, q, f, fo, qo, 1 << 30,
                            nullptr));
  EXPECT_ERR(moe_expert_ffn(ds, 65, MOE_REGIME_DECODE, q, f, ids, ids, q, f, q, f, q, f, fo, qo, 1 << 30, nullptr));
  EXPECT_ERR(moe_expert_ffn_w8a16(ds, 65, x, ids, ids, q, f, q, f, q, f, fo, qo, 1 << 30, nullptr));
  EXPECT_ERR(moe_expert_ffn_w8a16(ds, 4, x, ids, ids, q, f, q, f, q, f, fo, nullptr, 0, nullptr));
  EXPECT_ERR(moe_expert_ffn_w8a16(ds, -4, x, ids, ids, q, f, q, f, q, f, fo, qo, 1 << 30, nullptr));

  // combine
  EXPECT_ERR(moe_combine(nullptr, ids, f, 4, 8, 7168, xo, nullptr));
  EXPECT_ERR(moe_combine(f, ids, f, -1, 8, 7168, xo, nullptr));
  EXPECT_ERR(moe_combine(f, ids, f, 4, 0, 7168, xo, nullptr));
  EXPECT_ERR(moe_combine(f, ids, f, 4, 8, 7000, xo, nullptr));
  EXPECT_ERR(moe_combine(f, ids, f, INT32_MAX, 32, 7168, xo, nullptr));

  // whole layer, and the allocation-free entry point (stops before its scratch lookup)
  for (const moe_dims_t& d : kDims)
    for (moe_regime_t rg : kRegimes)
      for (int32_t T : {-1, 65, 4096, INT32_MAX}) {
        EXPECT_ERR(moe_ffn_layer(d, T, rg, x, ids, f, q, f, q, f, q, f, xo, io, nullptr, 0, nullptr));
        EXPECT_ERR(moe_ffn_layer_noalloc(d, T, rg, x, ids, f, q, f, q, f, q, f, xo, io, nullptr));
      }
  EXPECT(moe_ffn_layer(ds, 0, MOE_REGIME_AUTO, x, ids, f, q, f, q, f, q, f, xo, io, nullptr, 0, nullptr), MOE_OK);
  EXPECT(moe_ffn_layer(ds, 4, MOE_REGIME_AUTO, x, ids, f, q, f, q, f, q, f, xo, io, nullptr, 0, nullptr),
         MOE_ERR_WORKSPACE);
  EXPECT(moe_ffn_layer(ds, 4, MOE_REGIME_AUTO, x, ids, f, q, f, q, f, q, f, xo, io, qo + 8, 1u << 30, nullptr),
         MOE_ERR_INVALID_ARG);  // misaligned workspace
  EXPECT(moe_ffn_layer_noalloc(ds, 4096, MOE_REGIME_PREFILL, x, ids, f, q, f, q, f, q, f, xo, io, nullptr),
         MOE_ERR_WORKSPACE);  // beyond the scratch array
  EXPECT_ERR(moe_ffn_layer(ds, 4, MOE_REGIME_AUTO, x, ids, f, nullptr, f, q, f, q, f, xo, io, qo, 1u << 30,
                           nullptr));

  // router
  const moe_router_cfg_t cfg{8, 4, 2.5f, -1};
  for (int32_t E : {0, 7, 1025})
    EXPECT_ERR(moe_router(x, 4, 7168, x, f, E, 8, cfg, io, fo, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_router(x, 4, 7000, x, f, 256, 8, cfg, io, fo, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_router(x, 4, 7168, x, f, 256, 33, cfg, io, fo, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_router(x, 4, 7168, x, f, 256, 8, moe_router_cfg_t{3, 1, 1.f, -1}, io, fo, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_router(x, 4, 7168, x, f, 256, 8, moe_router_cfg_t{8, 9, 1.f, -1}, io, fo, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_router(x, 4, 7168, x, f, 256, 8, moe_router_cfg_t{8, 4, 0.f, -1}, io, fo, qo, 1 << 20, nullptr));
  EXPECT_ERR(moe_router(x, 4, 7168, x, f, 256, 8, cfg, io, fo, nullptr, 0, nullptr));
  EXPECT_ERR(moe_router(x, -4, 7168, x, f, 256, 8, cfg, io, fo, qo, 1 << 20, nullptr));

  // streamed layer (argument and shape errors come before the context is used)
  for (const moe_dims_t& d : kDims)
    for (int32_t T : {-1, 4096})
      for (int32_t chunk : {0, 1, 4096})
        EXPECT_ERR(moe_ffn_streamed(d, T, chunk, x, ids, f, q, f, q, f, q, f, qo, fo, nullptr, xo, io, qo, 1u << 30,
                                    nullptr, nullptr));
  moe_stream_ctx_t ctx = nullptr;
  EXPECT(moe_stream_ctx_create(0, &ctx), MOE_ERR_INVALID_ARG);
  EXPECT(moe_stream_ctx_create(5000, &ctx), MOE_ERR_INVALID_ARG);
  EXPECT(moe_stream_ctx_create(4, nullptr), MOE_ERR_INVALID_ARG);
  moe_stream_ctx_destroy(nullptr);

  // diagnostics
  EXPECT(moe_profile_begin(-1), MOE_ERR_INVALID_ARG);
  float ms = 0.f;
  const char* name = nullptr;
  EXPECT_ERR(moe_profile_get(-1, &ms, &name));
  EXPECT_ERR(moe_profile_get(0, nullptr, &name));
  std::printf("argument errors done\n");
}

void status_strings() {
  for (int s = -10; s <= 10; ++s) {
    const char* str = moe_status_string((moe_status_t)s);
    if (!str || !*str) {
      ++g_failures;
      std::printf("empty status string for %d\n", s);
    }
  }
  if (!moe_last_error()) {
    ++g_failures;
    std::printf("moe_last_error returned null\n");
  }
}

}  // namespace

int main() {
  workspace_queries();
  ring_schedules();
  argument_errors();
  status_strings();
  std::printf("%d checked calls, %d failures\n", g_calls, g_failures);
  return g_failures == 0 ? 0 : 1;
}
