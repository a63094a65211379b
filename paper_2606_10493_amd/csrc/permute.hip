// Token -> expert permutation: a stable counting sort of the flat slots
// f = t*k + j by expert id (tokens gated and sorted by expert into per-expert
// token lists, as in the standard expert-parallel workflow of the paper).
//
// A token lists each expert at most once, so within one expert the stable
// order by f is the order by token.  Each 256-token chunk therefore builds,
// in LDS, one 256-bit token mask per expert (4 x 64-bit words, set with an
// order-independent atomic OR).  The rank of (t, e) inside the chunk is the
// number of set bits below t in e's mask, so the scatter is exact and
// deterministic without any order-dependent atomics.
//
// Slots whose id is out of range, or repeats an earlier slot's id in the
// same token, are reported in the device status word and parked after all
// valid rows (positions expert_offsets[E] .. T*k-1, in slot order), so the
// outputs stay a bijection and every later index stays in bounds.
//
//   one chunk  (T <= 256): permute_small_kernel does count, scan and scatter
//              (layer_prologue_kernel: the same, beside the activation quantization).
//   several chunks: permute_count_kernel -> permute_scan_kernel -> permute_scatter_kernel.
#include "common.h"

namespace moe {

namespace {

constexpr int kChunk = 256;      // tokens per workgroup (one per thread)
constexpr int kMaxExperts = 1024;
constexpr int kMaxTopk = 32;

struct SlotCheck {
  int expert;
  uint32_t err;  // MOE_DEV_* bits, 0 if the slot is valid
};

// The ids of one chunk (up to kChunk tokens x k) staged in LDS with one
// coalesced pass, so the per-slot checks below read LDS, not global memory.
// 16 bits hold any valid id (E <= 1024); ids outside [0, E) become -1.
__device__ __forceinline__ void stage_ids(int16_t* sid, const int32_t* __restrict__ ids, int64_t chunk0, int64_t T,
                                          int k, int E) {
  const int64_t ntok = min((int64_t)kChunk, T - chunk0);
  const int n = ntok > 0 ? (int)(ntok * k) : 0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int32_t id = ids[chunk0 * k + i];
    sid[i] = (int16_t)((id >= 0 && id < E) ? id : -1);
  }
}

// Slot j of the chunk's token lt (ids in LDS, sid = the chunk's ids).
__device__ __forceinline__ SlotCheck check_slot(const int16_t* sid, int lt, int j, int k, int E) {
  const int16_t* row = sid + lt * k;
  SlotCheck r;
  r.expert = row[j];
  r.err = 0;
  if (r.expert < 0 || r.expert >= E) {  // staged as -1
    r.err = MOE_DEV_BAD_EXPERT_ID;
    return r;
  }
  for (int i = 0; i < j; ++i)
    if (row[i] == r.expert) r.err = MOE_DEV_DUP_EXPERT_ID;
  return r;
}

// Fill the per-expert token masks of one chunk; returns this thread's error bits.
__device__ __forceinline__ uint32_t build_masks(unsigned long long* mask, int* bad_count, const int16_t* sid,
                                                int64_t t, int64_t T, int k, int E) {
  uint32_t err = 0;
  if (t < T) {
    const unsigned long long bit = 1ull << (threadIdx.x & 63);
    const int word = threadIdx.x >> 6;
    for (int j = 0; j < k; ++j) {
      const SlotCheck s = check_slot(sid, threadIdx.x, j, k, E);
      if (s.err == 0) {
        atomicOr(&mask[s.expert * 4 + word], bit);
      } else {
        err |= s.err;
        atomicAdd(bad_count, 1);
      }
    }
  }
  return err;
}

// Rank of token lt (chunk-local) among the chunk's tokens routed to e.
__device__ __forceinline__ int rank_of(const unsigned long long* mask, int e, int lt) {
  const int word = lt >> 6;
  const unsigned long long below = (1ull << (lt & 63)) - 1ull;
  int r = __popcll(mask[e * 4 + word] & below);
  for (int w = 0; w < word; ++w) r += __popcll(mask[e * 4 + w]);
  return r;
}

__device__ __forceinline__ int rank_in_chunk(const unsigned long long* mask, int e) {
  return rank_of(mask, e, threadIdx.x);
}

__device__ __forceinline__ int mask_count(const unsigned long long* mask, int e) {
  return __popcll(mask[e * 4]) + __popcll(mask[e * 4 + 1]) + __popcll(mask[e * 4 + 2]) + __popcll(mask[e * 4 + 3]);
}

__device__ __forceinline__ void report(int32_t* dev_status, uint32_t err) {
  // Any-lane OR, then one atomic per wave.
  for (int m = 32; m >= 1; m >>= 1) err |= (uint32_t)__shfl_xor((int)err, m, 64);
  if (dev_status && err && (threadIdx.x & 63) == 0) atomicOr(dev_status, (int)err);
}

// Valid slots of this chunk go to base_e + rank; invalid ones, in slot order,
// to bad_base + running index (walked by one thread: the error path only).
__device__ __forceinline__ void scatter_chunk(const unsigned long long* mask, const int16_t* sid, int64_t chunk0,
                                              int64_t T, int k, int E, const int32_t* base_of_e, int32_t bad_base,
                                              int bad_count, int32_t* sorted_src, int32_t* dest_row) {
  const int64_t t = chunk0 + threadIdx.x;
  if (t < T) {
    const int64_t tb = t * k;
    for (int j = 0; j < k; ++j) {
      const SlotCheck s = check_slot(sid, threadIdx.x, j, k, E);
      if (s.err) continue;
      const int32_t p = base_of_e[s.expert] + rank_in_chunk(mask, s.expert);
      dest_row[tb + j] = p;
      sorted_src[p] = (int32_t)(tb + j);
    }
  }
  if (bad_count > 0 && threadIdx.x == 0) {
    int32_t p = bad_base;
    const int64_t t1 = min(T, chunk0 + kChunk);
    for (int64_t tt = chunk0; tt < t1; ++tt)
      for (int j = 0; j < k; ++j) {
        const SlotCheck s = check_slot(sid, (int)(tt - chunk0), j, k, E);
        if (!s.err) continue;
        dest_row[tt * k + j] = p;
        sorted_src[p] = (int32_t)(tt * k + j);
        ++p;
      }
  }
}

// One chunk (T <= 256): mask, scan and scatter in one workgroup.  Threads
// take slots, not tokens, so that a few tokens with k slots each (decode)
// spread over k * T threads instead of a serial loop in T threads.
__device__ __forceinline__ void permute_one_chunk(const int32_t* __restrict__ ids, int T, int k, int E,
                                                  int32_t* __restrict__ offsets, int32_t* __restrict__ sorted_src,
                                                  int32_t* __restrict__ dest_row, int32_t* __restrict__ dev_status) {
  __shared__ unsigned long long mask[kMaxExperts * 4];
  __shared__ int start[kMaxExperts];
  __shared__ int16_t sid[kChunk * kMaxTopk];
  __shared__ int tmp[4];
  __shared__ int bad_count;
  for (int i = threadIdx.x; i < E * 4; i += 256) mask[i] = 0ull;
  if (threadIdx.x == 0) bad_count = 0;
  stage_ids(sid, ids, 0, T, k, E);
  __syncthreads();
  const int n = T * k;
  uint32_t err = 0;
  for (int f = threadIdx.x; f < n; f += 256) {
    const int t = f / k, j = f - t * k;
    const SlotCheck sc = check_slot(sid, t, j, k, E);
    if (sc.err == 0) {
      atomicOr(&mask[sc.expert * 4 + (t >> 6)], 1ull << (t & 63));
    } else {
      err |= sc.err;
      atomicAdd(&bad_count, 1);
    }
  }
  __syncthreads();
  // Thread i owns experts 4i .. 4i+3 for the scan.
  int c[4], local = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * threadIdx.x + q;
    c[q] = (e < E) ? mask_count(mask, e) : 0;
    local += c[q];
  }
  int total_valid;
  int run = block_exclusive_scan(local, tmp, &total_valid);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * threadIdx.x + q;
    if (e < E) {
      start[e] = run;
      offsets[e] = run;
    }
    run += c[q];
  }
  if (threadIdx.x == 0) offsets[E] = total_valid;
  __syncthreads();
  for (int f = threadIdx.x; f < n; f += 256) {
    const int t = f / k, j = f - t * k;
    const SlotCheck sc = check_slot(sid, t, j, k, E);
    if (sc.err) continue;
    const int32_t p = start[sc.expert] + rank_of(mask, sc.expert, t);
    dest_row[f] = p;
    sorted_src[p] = f;
  }
  if (bad_count > 0 && threadIdx.x == 0) {  // error path: invalid slots in slot order after the valid rows
    int32_t p = total_valid;
    for (int f = 0; f < n; ++f) {
      const int t = f / k;
      const SlotCheck sc = check_slot(sid, t, f - t * k, k, E);
      if (!sc.err) continue;
      dest_row[f] = p;
      sorted_src[p] = f;
      ++p;
    }
  }
  report(dev_status, err);
}

// At most kTinySlots slots (decode batches): the same results as
// permute_one_chunk with two barriers and no loop whose trip count depends
// on the slot count.  Each slot gets a key: its id if valid, INT_MAX if not
// (or past the slots).  Slot f's stable position among the valid slots is the
// number of keys g with (key[g], g) < (key[f], f); an invalid slot goes after
// all valid ones, in slot order (a ballot prefix count); offsets[e] is the
// number of keys below e.  The counts read the 64 keys as 16 broadcast int4
// LDS loads, issued together.
constexpr int kTinySlots = 64;

__device__ __forceinline__ void permute_tiny(const int32_t* __restrict__ ids, int T, int k, int E,
                                             int32_t* __restrict__ offsets, int32_t* __restrict__ sorted_src,
                                             int32_t* __restrict__ dest_row, int32_t* __restrict__ dev_status) {
  __shared__ int sid[kTinySlots];
  __shared__ __attribute__((aligned(16))) int key[kTinySlots];
  const int n = T * k, tid = threadIdx.x;
  if (tid < kTinySlots) {
    int id = -1;
    if (tid < n) {
      const int32_t v = ids[tid];
      id = (v >= 0 && v < E) ? v : -1;
    }
    sid[tid] = id;
  }
  __syncthreads();
  uint32_t err = 0;
  bool valid = false;
  int me = INT_MAX;
  if (tid < n) {
    const int t = tid / k, j = tid - t * k;
    const int id = sid[tid];
    if (id < 0) {
      err = MOE_DEV_BAD_EXPERT_ID;
    } else {
      for (int i = 0; i < j; ++i)
        if (sid[t * k + i] == id) err = MOE_DEV_DUP_EXPERT_ID;
    }
    valid = err == 0;
    me = valid ? id : INT_MAX;
  }
  if (tid < kTinySlots) key[tid] = me;
  // Slots live in wave 0 (n <= 64): its ballots count valid and invalid slots.
  const unsigned long long vmask = __ballot(tid < n && valid);
  const unsigned long long bmask = __ballot(tid < n && !valid);
  __syncthreads();
  const int4* k4 = reinterpret_cast<const int4*>(key);
  if (tid < n) {
    int pos;
    if (valid) {
      pos = 0;
#pragma unroll
      for (int q = 0; q < kTinySlots / 4; ++q) {
        const int4 v = k4[q];
        const int g = 4 * q;
        pos += (v.x < me || (v.x == me && g < tid)) ? 1 : 0;
        pos += (v.y < me || (v.y == me && g + 1 < tid)) ? 1 : 0;
        pos += (v.z < me || (v.z == me && g + 2 < tid)) ? 1 : 0;
        pos += (v.w < me || (v.w == me && g + 3 < tid)) ? 1 : 0;
      }
    } else {
      pos = __popcll(vmask) + __popcll(bmask & ((1ull << tid) - 1ull));
    }
    dest_row[tid] = pos;
    sorted_src[pos] = tid;
  }
  for (int e = tid; e < E; e += blockDim.x) {
    int c = 0;
#pragma unroll
    for (int q = 0; q < kTinySlots / 4; ++q) {
      const int4 v = k4[q];
      c += (v.x < e ? 1 : 0) + (v.y < e ? 1 : 0) + (v.z < e ? 1 : 0) + (v.w < e ? 1 : 0);
    }
    offsets[e] = c;
  }
  if (tid == 0) offsets[E] = __popcll(vmask);
  report(dev_status, err);
}

__global__ __launch_bounds__(256) void permute_small_kernel(const int32_t* __restrict__ ids, int T, int k, int E,
                                                            int32_t* __restrict__ offsets,
                                                            int32_t* __restrict__ sorted_src,
                                                            int32_t* __restrict__ dest_row,
                                                            int32_t* __restrict__ dev_status) {
  if (T * k <= kTinySlots) permute_tiny(ids, T, k, E, offsets, sorted_src, dest_row, dev_status);
  else permute_one_chunk(ids, T, k, E, offsets, sorted_src, dest_row, dev_status);
}

// Layer prologue for one chunk of tokens (T <= 256), one launch instead of
// two: workgroup 0 sorts the slots (as permute_small_kernel); workgroups 1..
// quantize the bf16 activations, 16 groups of 128 columns each (as
// moe_quant_act).
__global__ __launch_bounds__(256) void layer_prologue_kernel(const int32_t* __restrict__ ids, int T, int k, int E,
                                                             int32_t* __restrict__ offsets,
                                                             int32_t* __restrict__ sorted_src,
                                                             int32_t* __restrict__ dest_row,
                                                             int32_t* __restrict__ dev_status,
                                                             const uint16_t* __restrict__ x, int64_t n_groups,
                                                             int groups_per_row, uint8_t* __restrict__ qx,
                                                             float* __restrict__ sx) {
  if (blockIdx.x == 0) {
    if (T * k <= kTinySlots) permute_tiny(ids, T, k, E, offsets, sorted_src, dest_row, dev_status);
    else permute_one_chunk(ids, T, k, E, offsets, sorted_src, dest_row, dev_status);
    return;
  }
  const int64_t g = (int64_t)(blockIdx.x - 1) * 16 + (threadIdx.x >> 4);
  if (g >= n_groups) return;  // whole 16-lane groups leave together
  quant_row_group<uint16_t>(x, g, threadIdx.x & 15, groups_per_row, qx, sx);
}

// counts: [n_chunks][E+1]; entry E is the chunk's number of invalid slots.
__global__ __launch_bounds__(256) void permute_count_kernel(const int32_t* __restrict__ ids, int T, int k, int E,
                                                            int32_t* __restrict__ counts,
                                                            int32_t* __restrict__ dev_status) {
  __shared__ unsigned long long mask[kMaxExperts * 4];
  __shared__ int16_t sid[kChunk * kMaxTopk];
  __shared__ int bad_count;
  for (int i = threadIdx.x; i < E * 4; i += 256) mask[i] = 0ull;
  if (threadIdx.x == 0) bad_count = 0;
  const int64_t chunk0 = (int64_t)blockIdx.x * kChunk;
  stage_ids(sid, ids, chunk0, T, k, E);
  __syncthreads();
  const uint32_t err = build_masks(mask, &bad_count, sid, chunk0 + threadIdx.x, T, k, E);
  __syncthreads();
  int32_t* row = counts + (int64_t)blockIdx.x * (E + 1);
  for (int e = threadIdx.x; e < E; e += 256) row[e] = mask_count(mask, e);
  if (threadIdx.x == 0) row[E] = bad_count;
  report(dev_status, err);
}

// One workgroup of 1024 threads; thread e scans expert e over the chunks.
__global__ __launch_bounds__(1024) void permute_scan_kernel(const int32_t* __restrict__ counts, int n_chunks, int E,
                                                            int32_t* __restrict__ base,
                                                            int32_t* __restrict__ offsets) {
  __shared__ int wave_tot[16];
  const int e = threadIdx.x;
  int tot = 0;
  // Unrolled by 8 so that eight independent loads go out before the first
  // wait (a plain loop waited for every chunk's count in turn).
  if (e < E) {
#pragma unroll 8
    for (int c = 0; c < n_chunks; ++c) tot += counts[(int64_t)c * (E + 1) + e];
  }
  int total_valid;
  const int excl = block_exclusive_scan(tot, wave_tot, &total_valid);
  if (e < E) {
    int run = excl;
    offsets[e] = run;
#pragma unroll 8
    for (int c = 0; c < n_chunks; ++c) {
      const int64_t i = (int64_t)c * (E + 1) + e;
      base[i] = run;
      run += counts[i];
    }
  }
  if (e == 0) {
    offsets[E] = total_valid;
    int run = total_valid;
    for (int c = 0; c < n_chunks; ++c) {
      const int64_t i = (int64_t)c * (E + 1) + E;
      base[i] = run;
      run += counts[i];
    }
  }
}

__global__ __launch_bounds__(256) void permute_scatter_kernel(const int32_t* __restrict__ ids, int T, int k, int E,
                                                              const int32_t* __restrict__ counts,
                                                              const int32_t* __restrict__ base,
                                                              int32_t* __restrict__ sorted_src,
                                                              int32_t* __restrict__ dest_row) {
  __shared__ unsigned long long mask[kMaxExperts * 4];
  __shared__ int16_t sid[kChunk * kMaxTopk];
  __shared__ int bad_count;
  for (int i = threadIdx.x; i < E * 4; i += 256) mask[i] = 0ull;
  if (threadIdx.x == 0) bad_count = 0;
  const int64_t chunk0 = (int64_t)blockIdx.x * kChunk;
  stage_ids(sid, ids, chunk0, T, k, E);
  __syncthreads();
  build_masks(mask, &bad_count, sid, chunk0 + threadIdx.x, T, k, E);
  __syncthreads();
  const int32_t* brow = base + (int64_t)blockIdx.x * (E + 1);
  const int nbad = counts[(int64_t)blockIdx.x * (E + 1) + E];
  scatter_chunk(mask, sid, chunk0, T, k, E, brow, brow[E], nbad, sorted_src, dest_row);
}

int64_t n_chunks_of(int32_t T) { return ((int64_t)T + kChunk - 1) / kChunk; }

}  // namespace

// Quantize x [T, H] and sort the slots of T <= 256 tokens in one launch.
// Arguments are checked by the caller.
moe_status_t launch_layer_prologue(const uint16_t* x, int32_t T, int32_t H, const int32_t* topk_ids, int32_t k,
                                   int32_t E, uint8_t* qx, float* sx, int32_t* offsets, int32_t* sorted_src,
                                   int32_t* dest_row, int32_t* dev_status, hipStream_t stream) {
  if (T > kChunk) return fail(MOE_ERR_INVALID_ARG, "layer prologue: T=%d > %d", T, kChunk);
  const int gpr = H / kBlock;
  const int64_t n_groups = (int64_t)T * gpr;
  const int64_t blocks = 1 + (n_groups + 15) / 16;
  MOE_LAUNCH("layer_prologue", layer_prologue_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, topk_ids, T, k, E,
             offsets, sorted_src, dest_row, dev_status, x, n_groups, gpr, qx, sx);
  return check_launch("layer prologue");
}

}  // namespace moe

using namespace moe;

extern "C" size_t moe_permute_workspace(int32_t T, int32_t k, int32_t E) {
  (void)k;
  if (T < 0 || E <= 0) return 0;
  const int64_t nc = n_chunks_of(T);
  if (nc <= 1) return 256;
  return (size_t)(2 * nc * (E + 1) * sizeof(int32_t) + 256);
}

extern "C" moe_status_t moe_permute(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                                    int32_t* expert_offsets, int32_t* sorted_src, int32_t* dest_row,
                                    int32_t* dev_status, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (T < 0 || E < 1 || E > kMaxExperts || k < 1 || k > kMaxTopk || k > E)
    return fail(MOE_ERR_INVALID_ARG, "moe_permute: T=%d k=%d E=%d (need T>=0, 1<=k<=min(E,32), 1<=E<=1024)", T, k,
                E);
  if ((int64_t)T * k > 0x7fffffff) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "moe_permute: T*k overflows int32");
  if (!expert_offsets || (T > 0 && (!topk_ids || !sorted_src || !dest_row)))
    return fail(MOE_ERR_INVALID_ARG, "moe_permute: null pointer");
  const int64_t nc = n_chunks_of(T);
  if (nc <= 1) {
    MOE_LAUNCH("permute_small", permute_small_kernel, dim3(1), dim3(256), 0, stream, topk_ids, T, k, E, expert_offsets,
                       sorted_src, dest_row, dev_status);
    return check_launch("moe_permute");
  }
  const size_t need = moe_permute_workspace(T, k, E);
  if (!ws || ws_bytes < need)
    return fail(MOE_ERR_WORKSPACE, "moe_permute: workspace %zu bytes < %zu", ws_bytes, need);
  if (!aligned(ws, 4)) return fail(MOE_ERR_INVALID_ARG, "moe_permute: misaligned workspace");
  int32_t* counts = static_cast<int32_t*>(ws);
  int32_t* base = counts + nc * (E + 1);
  MOE_LAUNCH("permute_count", permute_count_kernel, dim3((unsigned)nc), dim3(256), 0, stream, topk_ids, T, k, E, counts,
                     dev_status);
  MOE_LAUNCH("permute_scan", permute_scan_kernel, dim3(1), dim3(1024), 0, stream, counts, (int)nc, E, base,
                     expert_offsets);
  MOE_LAUNCH("permute_scatter", permute_scatter_kernel, dim3((unsigned)nc), dim3(256), 0, stream, topk_ids, T, k, E, counts,
                     base, sorted_src, dest_row);
  return check_launch("moe_permute");
}
