// One routed-expert layer through the C ABI alone: HIP runtime calls and
// include/moe.h, no Python and no torch.  Used by tests/test_gpu_c_abi.py.
//
//   abi_c_layer H I E K T regime in_dir out_dir
//
// in_dir holds raw little-endian arrays: x.bin (bf16 bits [T, H]), ids.bin
// (int32 [T, K]), wts.bin (fp32 [T, K]), wg.bin, wu.bin (fp32 [E, I, H]),
// wd.bin (fp32 [E, H, I]).  The program allocates device memory, quantizes
// and packs the weights (moe_quant_weight, moe_pack_weight), runs the layer
// once through moe_ffn_layer and once through the four calls (moe_quant_act,
// moe_permute, moe_expert_ffn, moe_combine) on a stream of its own, and
// writes out_fused.bin and out_calls.bin (bf16 bits [T, H]) to out_dir.
// Exit status 0 on success; any failed call prints the library's message.
#include <hip/hip_runtime_api.h>

#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "moe.h"

namespace {

int fail_hip(hipError_t e, const char* what) {
  std::fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
  return 2;
}

#define HIP_OK(call)                              \
  do {                                            \
    const hipError_t e_ = (call);                 \
    if (e_ != hipSuccess) return fail_hip(e_, #call); \
  } while (0)

#define MOE_OK_OR_FAIL(call)                                                                      \
  do {                                                                                            \
    const moe_status_t s_ = (call);                                                               \
    if (s_ != MOE_OK) {                                                                           \
      std::fprintf(stderr, "%s: %s (%s)\n", #call, moe_status_string(s_), moe_last_error());      \
      return 3;                                                                                   \
    }                                                                                             \
  } while (0)

template <typename T>
bool read_file(const std::string& path, std::vector<T>& out, size_t n) {
  out.resize(n);
  FILE* f = std::fopen(path.c_str(), "rb");
  if (!f) return false;
  const size_t got = std::fread(out.data(), sizeof(T), n, f);
  std::fclose(f);
  return got == n;
}

template <typename T>
bool write_file(const std::string& path, const std::vector<T>& v) {
  FILE* f = std::fopen(path.c_str(), "wb");
  if (!f) return false;
  const size_t put = std::fwrite(v.data(), sizeof(T), v.size(), f);
  std::fclose(f);
  return put == v.size();
}

template <typename T>
int to_device(const std::vector<T>& h, T** d) {
  HIP_OK(hipMalloc(reinterpret_cast<void**>(d), h.size() * sizeof(T) + 16));
  HIP_OK(hipMemcpy(*d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
  return 0;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 9) {
    std::fprintf(stderr, "usage: %s H I E K T regime in_dir out_dir\n", argv[0]);
    return 1;
  }
  const int32_t H = std::atoi(argv[1]), I = std::atoi(argv[2]), E = std::atoi(argv[3]), K = std::atoi(argv[4]),
                T = std::atoi(argv[5]);
  const moe_regime_t regime = (moe_regime_t)std::atoi(argv[6]);
  const std::string in = argv[7], out = argv[8];
  const moe_dims_t d{H, I, E, K};

  std::vector<uint16_t> x;
  std::vector<int32_t> ids;
  std::vector<float> wts, wg, wu, wd;
  if (!read_file(in + "/x.bin", x, (size_t)T * H) || !read_file(in + "/ids.bin", ids, (size_t)T * K) ||
      !read_file(in + "/wts.bin", wts, (size_t)T * K) || !read_file(in + "/wg.bin", wg, (size_t)E * I * H) ||
      !read_file(in + "/wu.bin", wu, (size_t)E * I * H) || !read_file(in + "/wd.bin", wd, (size_t)E * H * I)) {
    std::fprintf(stderr, "cannot read the inputs in %s\n", in.c_str());
    return 1;
  }

  hipStream_t stream;
  HIP_OK(hipStreamCreateWithFlags(&stream, hipStreamNonBlocking));

  uint16_t* dx;
  int32_t* dids;
  float* dwts;
  if (to_device(x, &dx) || to_device(ids, &dids) || to_device(wts, &dwts)) return 2;

  // Weights: fp32 -> e4m3 codes + 128x128 scales -> operand-tile packing.
  uint8_t* q[3];
  float* s[3];
  {
    const std::vector<float>* w[3] = {&wg, &wu, &wd};
    const int32_t rows[3] = {I, I, H}, cols[3] = {H, H, I};
    for (int m = 0; m < 3; ++m) {
      float* dw;
      uint8_t* raw;
      if (to_device(*w[m], &dw)) return 2;
      const size_t n = (size_t)E * rows[m] * cols[m];
      HIP_OK(hipMalloc(reinterpret_cast<void**>(&raw), n));
      HIP_OK(hipMalloc(reinterpret_cast<void**>(&q[m]), n));
      HIP_OK(hipMalloc(reinterpret_cast<void**>(&s[m]), (size_t)E * (rows[m] / 128) * (cols[m] / 128) * sizeof(float)));
      MOE_OK_OR_FAIL(moe_quant_weight(dw, E, rows[m], cols[m], raw, s[m], stream));
      MOE_OK_OR_FAIL(moe_pack_weight(raw, E, rows[m], cols[m], q[m], stream));
      HIP_OK(hipStreamSynchronize(stream));
      HIP_OK(hipFree(dw));
      HIP_OK(hipFree(raw));
    }
  }

  int32_t* status;
  HIP_OK(hipMalloc(reinterpret_cast<void**>(&status), sizeof(int32_t)));
  HIP_OK(hipMemsetAsync(status, 0, sizeof(int32_t), stream));
  uint16_t* dout;
  HIP_OK(hipMalloc(reinterpret_cast<void**>(&dout), (size_t)T * H * sizeof(uint16_t)));
  std::vector<uint16_t> host_out((size_t)T * H);

  // 1. The whole layer in one call.
  {
    const size_t ws_bytes = moe_ffn_layer_workspace(d, T, regime);
    void* ws;
    HIP_OK(hipMalloc(&ws, ws_bytes > 0 ? ws_bytes : 256));
    MOE_OK_OR_FAIL(moe_ffn_layer(d, T, regime, dx, dids, dwts, q[0], s[0], q[1], s[1], q[2], s[2], dout, status,
                                 ws, ws_bytes, stream));
    HIP_OK(hipMemcpyAsync(host_out.data(), dout, host_out.size() * sizeof(uint16_t), hipMemcpyDeviceToHost, stream));
    HIP_OK(hipStreamSynchronize(stream));
    HIP_OK(hipFree(ws));
    if (!write_file(out + "/out_fused.bin", host_out)) return 1;
  }

  // 2. The four calls.
  {
    const size_t R = (size_t)T * K;
    uint8_t* qx;
    float *sx, *y;
    int32_t *offsets, *sorted_src, *dest_row;
    HIP_OK(hipMalloc(reinterpret_cast<void**>(&qx), (size_t)T * H));
    HIP_OK(hipMalloc(reinterpret_cast<void**>(&sx), (size_t)T * (H / 128) * sizeof(float)));
    HIP_OK(hipMalloc(reinterpret_cast<void**>(&offsets), (size_t)(E + 1) * sizeof(int32_t)));
    HIP_OK(hipMalloc(reinterpret_cast<void**>(&sorted_src), R * sizeof(int32_t)));
    HIP_OK(hipMalloc(reinterpret_cast<void**>(&dest_row), R * sizeof(int32_t)));
    HIP_OK(hipMalloc(reinterpret_cast<void**>(&y), R * H * sizeof(float)));
    const size_t pws_bytes = moe_permute_workspace(T, K, E), fws_bytes = moe_expert_ffn_workspace(d, T, regime);
    void *pws, *fws;
    HIP_OK(hipMalloc(&pws, pws_bytes > 0 ? pws_bytes : 256));
    HIP_OK(hipMalloc(&fws, fws_bytes > 0 ? fws_bytes : 256));
    MOE_OK_OR_FAIL(moe_quant_act(dx, T, H, qx, sx, stream));
    MOE_OK_OR_FAIL(moe_permute(dids, T, K, E, offsets, sorted_src, dest_row, status, pws, pws_bytes, stream));
    MOE_OK_OR_FAIL(moe_expert_ffn(d, T, regime, qx, sx, offsets, sorted_src, q[0], s[0], q[1], s[1], q[2], s[2], y,
                                  fws, fws_bytes, stream));
    MOE_OK_OR_FAIL(moe_combine(y, dest_row, dwts, T, K, H, dout, stream));
    HIP_OK(hipMemcpyAsync(host_out.data(), dout, host_out.size() * sizeof(uint16_t), hipMemcpyDeviceToHost, stream));
    int32_t st = -1;
    HIP_OK(hipMemcpyAsync(&st, status, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
    HIP_OK(hipStreamSynchronize(stream));
    if (st != 0) {
      std::fprintf(stderr, "device status %d\n", st);
      return 4;
    }
    if (!write_file(out + "/out_calls.bin", host_out)) return 1;
    for (void* p : {(void*)qx, (void*)sx, (void*)y, (void*)offsets, (void*)sorted_src, (void*)dest_row, pws, fws})
      HIP_OK(hipFree(p));
  }

  for (int m = 0; m < 3; ++m) {
    HIP_OK(hipFree(q[m]));
    HIP_OK(hipFree(s[m]));
  }
  for (void* p : {(void*)dx, (void*)dids, (void*)dwts, (void*)status, (void*)dout}) HIP_OK(hipFree(p));
  HIP_OK(hipStreamDestroy(stream));
  std::printf("layer through the C ABI: T=%d H=%d I=%d E=%d k=%d regime=%d done\n", T, H, I, E, K, (int)regime);
  return 0;
}
