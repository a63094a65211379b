// Prefill-regime expert FFN: block-scaled FP8 MFMA grouped GEMM over the
// expert-sorted rows (the GPU FP8 GEMM path of the paper's FP8 Block Scaling
// Format: FP8 weights and scales from device memory, activations quantized
// to FP8, FP8 x FP8 products with FP32 accumulation; gate and up fused with
// SiLU(gate)*up as in the paper's stage one, down after it).
//
// The products are formed transposed, D = W x X^T, with the MFMA 32x32x64:
// its A operand is 32 weight rows (output channels), its B operand 32
// expert rows (tokens), two instructions per 128-K scale block.  A lane's
// 16 results then share one token and lie inside one 128-channel weight-
// scale block (GATEUP: eight gate, eight up), so the per-block scale of a
// result is (the lane's token scale) x (a wave-uniform weight scale), and
// the promotion into the fp32 accumulators costs 16 FMAs per two MFMAs: few
// enough VALU operations for the matrix core to stay busy (measured on
// gfx950: up to about 9 independent VALU operations per 32x32x64 MFMA issue
// alongside it at full rate, against 4 per 16x16x128).
//
// Tile: 256 weight rows x 128 expert rows x one 128-K block per step, 512
// threads (8 waves).  Wave w owns 32 weight rows against all 128 expert rows
// (four B operands): 8 MFMA per K step.  The weights are packed in operand
// tiles (moe_pack_weight), so they go from global memory straight into the
// MFMA operand registers with 1 KB-contiguous wave loads (no wave shares
// them), through a ring of kRing K blocks loaded kRing - 1 steps ahead.
// Only the expert rows, which all waves read, are staged through LDS
// (three stages, 16-byte chunks XOR-swizzled by row) and their scales sit
// in LDS transposed, [K block][row].  Waves 0-3 and 4-7 run the K loop half
// a step apart (a memory phase and a compute phase per step, a barrier after
// each), so that on every SIMD one wave feeds the matrix core while the
// other loads: with all eight waves in step, both waves of a SIMD wait for
// LDS together and then queue for the matrix core together.
//
// GATEUP: wave w's rows are gate rows nt*128 + 16w + [0, 16) followed by the
// same up rows, so a workgroup holds one full 128-wide block of h: its
// epilogue computes h = SiLU(G) * U, the per-row amax of the block (lanes,
// then the eight waves through LDS), the scale sh = amax / 448 and the e4m3
// codes qh, staged through LDS and written as 16-byte rows.
// DOWN: wave w's rows are W_down rows nt*256 + 32w + [0, 32); the epilogue
// writes fp32 in 16-byte pieces.
//
// Work items are (expert m-tile, n-tile) pairs; m-tiles of all experts are
// numbered by an exclusive scan of ceil(M_e / 128) and described one by one
// (prefill_tiles_kernel), so a workgroup finds its tile with one load,
// an expert's 32-row groups are dealt evenly over its m-tiles, and its
// items are ordered n-tile major, so the m-tiles sharing a weight slice are
// neighbours of similar size.  Work items are assigned XCD-major: the
// hardware deals workgroups to the 8 XCDs round-robin, so with n real items
// (read from the tile scan; the grid is only an upper bound) item = (block
// % 8) * ceil(n / 8) + block / 8 keeps an expert's items on one XCD's L2
// while every XCD gets an equal share.
#include "common.h"

#include <type_traits>

namespace moe {

namespace {

constexpr int kBM = 128;                // expert rows (tokens) per tile
constexpr int kBN = 256;                // weight rows per tile
constexpr int kThreads = 512;           // 8 waves x 32 weight rows
constexpr int kLdsRow = kBlock;         // LDS row (bytes); 16-byte chunks XOR-swizzled, see swz()
constexpr int kHalf = kBM * kLdsRow;    // one K block of the expert rows (one LDS stage)
constexpr int kStages = 3;              // LDS stages of the ping-pong pipeline
constexpr int kSaStride = kBM + 1;      // floats per K block of the row-scale table
constexpr int kRing = 3;                // weight K blocks in registers
constexpr int kXcd = 8;
constexpr int kBand = 8;                // m-tiles per band of the work-item order (see tile_of)

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

struct PrefillArgs {
  const uint8_t* a;           // e4m3 activations [a_rows, K]
  const float* sa;            // [a_rows, K/128]
  const int32_t* sorted_src;  // GATEUP without row tables: A row of sorted row p = sorted_src[p] / topk; else unused
  const int32_t* row_pos;     // NULL: tile rows are sorted positions; else the sorted position of launch row v
  const int32_t* row_tok;     // GATEUP with row_pos: the token (A row) of launch row v
  int topk;
  int a_rows;
  const int32_t* mtile_start; // [n_units+1] exclusive scan of the experts' m-tile counts
  const int4* desc;           // [max_mtiles] m-tile block descriptors (prefill_tiles_kernel)
  int64_t max_mtiles;         // bound on the m-tiles (sizes desc)
  int n_units;                // experts of the launch
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

// The rows of a launch.  One chunk (a resident layer): expert u owns the
// sorted positions [offsets[u], offsets[u+1]).  Several chunks, each sorted
// on its own (chunk c's positions start at c * chunk_rows, its offsets at
// offsets + c * off_stride): expert u owns M_u = the sum of its rows over
// the chunks, numbered as launch rows [vstart[u], vstart[u] + M_u) in chunk
// order (prefill_rows_kernel maps each launch row to its sorted position and
// token), so the tiles of an expert span chunks and all of them read the
// expert's weight slices together.  mtile_start = exclusive scan of the
// experts' m-tile counts ceil(M_u / 128), and for every m-tile index b in
// [mtile_start[u], mtile_start[u+1]) desc[b] = (u, mtile_start[u], first
// row, end row), from which a GEMM workgroup derives its tile with one
// uniform load (no search).  Experts are taken 1024 at a time with running
// totals.
__global__ __launch_bounds__(1024) void prefill_tiles_kernel(const int32_t* __restrict__ offsets, int64_t off_stride,
                                                             int n_units, int n_chunks,
                                                             int32_t* __restrict__ mtile_start,
                                                             int32_t* __restrict__ vstart,
                                                             int4* __restrict__ desc, int64_t max_mtiles) {
  __shared__ int wave_tot[16];
  int carry_t = 0, carry_v = 0;
  for (int base = 0; base < n_units; base += 1024) {
    const int u = base + (int)threadIdx.x;
    int o0 = 0, m = 0;
    if (u < n_units) {
      if (n_chunks == 1) {
        o0 = offsets[u];
        m = offsets[u + 1] - o0;
      } else {
        for (int c = 0; c < n_chunks; ++c) m += offsets[c * off_stride + u + 1] - offsets[c * off_stride + u];
      }
    }
    const int cnt = m > 0 ? (m + kBM - 1) / kBM : 0;
    int tot_t, tot_v;
    const int excl = carry_t + block_exclusive_scan(cnt, wave_tot, &tot_t);
    const int v0 = carry_v + block_exclusive_scan(m, wave_tot, &tot_v);
    if (n_chunks > 1) o0 = v0;
    if (u < n_units) {
      mtile_start[u] = excl;
      vstart[u] = v0;
    }
    for (int b = excl; b < excl + cnt && b < max_mtiles; ++b) desc[b] = make_int4(u, excl, o0, o0 + m);
    carry_t += tot_t;
    carry_v += tot_v;
  }
  if (threadIdx.x == 0) {
    mtile_start[n_units] = carry_t;
    vstart[n_units] = carry_v;
  }
}

// Row tables of a launch over several chunks: block (c, u) writes the
// launch rows of expert u's rows in chunk c, in order: row_pos = the sorted
// position, row_tok = the token (the chunk-relative slot / topk plus the
// chunk's first token).
__global__ __launch_bounds__(256) void prefill_rows_kernel(const int32_t* __restrict__ offsets, int64_t off_stride,
                                                           int64_t chunk_rows, int chunk_tokens,
                                                           const int32_t* __restrict__ sorted_src, int topk,
                                                           const int32_t* __restrict__ vstart,
                                                           int32_t* __restrict__ row_pos,
                                                           int32_t* __restrict__ row_tok) {
  const int c = blockIdx.x, u = blockIdx.y;
  int v = vstart[u];
  for (int cc = 0; cc < c; ++cc) v += offsets[cc * off_stride + u + 1] - offsets[cc * off_stride + u];
  const int p0 = offsets[c * off_stride + u];
  const int cnt = offsets[c * off_stride + u + 1] - p0;
  const int64_t base = (int64_t)c * chunk_rows + p0;
  for (int r = threadIdx.x; r < cnt; r += blockDim.x) {
    const int64_t pos = base + r;
    row_pos[v + r] = (int32_t)pos;
    row_tok[v + r] = sorted_src[pos] / topk + c * chunk_tokens;
  }
}

// The tiles workspace: mtile_start [n_units+1], vstart [n_units+1] (each
// padded to 16 bytes), desc [max_mtiles]; with several chunks also row_pos
// and row_tok [rows] each.
size_t tiles_index_bytes(int64_t n_units) { return ((size_t)(n_units + 1) * sizeof(int32_t) + 15) & ~(size_t)15; }
size_t tiles_desc_offset(int64_t n_units) { return 2 * tiles_index_bytes(n_units); }

// LDS byte offset of 16-byte chunk c (0..7) of row `row` in a 128-byte-row
// tile.  gfx950's LDS serves 256 bytes per clock (64 four-byte banks), so
// two consecutive 128-byte rows share one bank row; the chunk index is
// XOR-ed with (row / 2) % 8, so the 16 rows that a quarter-wave b128 read
// touches fill all 16 sixteen-byte bank slots (measured on gfx950: about
// 195 B/clk per CU this way, 122 with the chunk XOR-ed by row % 8, whose
// rows r and r + 8 collide, and 32 unswizzled).
__device__ __forceinline__ int swz(int row, int c) { return row * kLdsRow + ((c ^ ((row >> 1) & 7)) << 4); }

__device__ __forceinline__ v16f mfma_f8_32x32x64(const v8i& a, const v8i& b, const v16f& c) {
  // Scale operands 0: the compiler emits the unscaled v_mfma_f32_32x32x64_f8f6f4
  // (e4m3 operands, no block scales; see mfma_f8_16x16x128).
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// The tile of work item `item`: expert u owns items [mtile_start[u],
// mtile_start[u+1]) * n_tiles, in bands of kBand consecutive m-tiles, each
// band n-tile major: item = mtile_start[u] * n_tiles + kBand * n_tiles *
// band + nt * width + (mt - kBand * band) (width = the band's m-tiles; an
// expert with at most kBand m-tiles is one band).  The m-tiles that read the
// same weight slice (same nt) are neighbours, so they run together on one
// XCD and the slice comes from HBM once per band (m-tile major order
// fetched the weights once per m-tile); and an expert with many m-tiles
// re-reads its token rows once per band pass instead of once per n-tile
// (one n-tile-major pass over 141 m-tiles evicts them from L2 before the
// next n-tile reads them again).  The expert's ceil(M/32) row groups are dealt evenly over its
// mcount tiles (tile mt gets q/mcount groups, one more for mt < q % mcount):
// the same MFMA work as full tiles plus a tail, but tiles of similar size,
// which advance through their shared weight slice at similar speed, so the
// slice is fetched from HBM once and read by the others from L2 (a 1-32-row
// tail tile ran about 3.6 times faster than the full tiles and fetched the
// slice ahead of them; gate/up read 1.7 times its algorithmic bytes).
struct Tile {
  int e, m0, mc, nt;  // expert, first row (a sorted position, or a launch row with row tables), rows, n-tile
};

__device__ __forceinline__ Tile tile_of(const PrefillArgs& p, int item) {
  const int4 d = p.desc[item / p.n_tiles];
  const int e = d.x, s0 = d.y, o0 = d.z, o1 = d.w;
  const int mcount = (o1 - o0 + kBM - 1) / kBM;
  const int local = item - s0 * p.n_tiles;
  const int band = local / (kBand * p.n_tiles);
  const int bw = min(kBand, mcount - band * kBand);
  const int in_band = local - band * kBand * p.n_tiles;
  const int ntx = in_band / bw;
  const int mt = band * kBand + (in_band - ntx * bw);
  const int q = (o1 - o0 + 31) >> 5;
  const int base = q / mcount, extra = q - base * mcount;
  const int first = o0 + 32 * (mt * base + min(mt, extra));
  const int groups = base + (mt < extra ? 1 : 0);
  return Tile{e, first, min(32 * groups, o1 - first), ntx};
}

template <bool GATEUP>
__global__ __launch_bounds__(kThreads) void ffn_prefill_kernel(PrefillArgs p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  __shared__ int arow[kBM];   // A row (token for GATEUP, sorted position for DOWN) of tile row t, -1 if none
  __shared__ int orow[kBM];   // sorted position (output row) of tile row t < mc
  __shared__ float rowmax[8][kBM];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r32 = lane & 31;  // operand row (A) / column (B) of this lane
  const int g2 = lane >> 5;   // K half of a 64-K MFMA slice this lane supplies

  // XCD-major work item over the real items (the grid is an upper bound):
  // XCD x takes items [x*per, (x+1)*per) in order.
  int total = p.mtile_start[p.n_units];
  if (total > p.max_mtiles) total = (int)p.max_mtiles;  // inconsistent offsets: only described m-tiles run
  const int real = total * p.n_tiles;  // < 2^31 (the grid bound is checked on the host)
  const int per = (real + kXcd - 1) / kXcd;
  const int slot = blockIdx.x / kXcd;
  if (slot >= per) return;
  const int item = (int)(blockIdx.x % kXcd) * per + slot;
  if (item >= real) return;
  const Tile tile = tile_of(p, item);  // one uniform load, no search and no barrier
  const int m0 = tile.m0;  // first sorted row of the tile
  const int mc = tile.mc;  // rows in the tile
  const int nt = tile.nt;  // n-tile
  const int nb = p.K / kBlock;

  float* sa_lds = reinterpret_cast<float*>(smem + kStages * kHalf);  // [nb][kSaStride]
  float* sw_lds = sa_lds + nb * kSaStride;                       // [2][nb]

  // This wave's 32-row weight operand: rows 0-15 and 16-31 are two packed
  // 16-row groups (GATEUP: the gate and the up group nt*8 + w; DOWN: groups
  // nt*16 + 2w and + 1).  Lane l reads row l % 32, K bytes 64h + 32 g2 +
  // [0, 32) of each block, i.e. kq = 2 g2 and 2 g2 + 1 of the packed tile.
  const uint8_t* wsrc;
  {
    const int64_t ebase = (int64_t)tile.e * p.N * p.K;
    const int64_t grp = GATEUP ? (int64_t)nt * (kBlock / 16) + wave : (int64_t)nt * (kBN / 16) + 2 * wave + (r32 >> 4);
    const uint8_t* wm = (GATEUP && r32 >= 16) ? p.w1 : p.w0;
    wsrc = wm + ebase + grp * nb * kTileBytes + packed_lane_offset(0, 2 * g2, r32 & 15);
  }
  v8i wr[kRing][2];  // [slot][K half]
#define MOE_PF_WLOAD(SLOT, BLK)                                                            \
  do {                                                                                     \
    const uint8_t* w_ = wsrc + (int64_t)(BLK) * kTileBytes;                                \
    wr[SLOT][0] = join_v8i(*reinterpret_cast<const uint4*>(w_),                            \
                           *reinterpret_cast<const uint4*>(w_ + 512));                     \
    wr[SLOT][1] = join_v8i(*reinterpret_cast<const uint4*>(w_ + 1024),                     \
                           *reinterpret_cast<const uint4*>(w_ + 1536));                    \
  } while (0)

  // The set-up before the first MFMA is two round trips after the tile
  // lookup: (1) the row indices and weight scales, with the first two
  // weight blocks issued behind them; (2) the row scales and the first two K
  // blocks of expert rows (the weights are in flight since round trip 1).
  // Each load loop is written so that a thread issues all its loads before
  // it waits for any.  Weight scales of the tile's two 128-row blocks:
  // GATEUP gate and up block nt; DOWN blocks 2nt and 2nt + 1 (waves 0-3 and
  // 4-7).
  auto issue_indices_and_weights = [&]() {
    // One unconditional 4-byte load per thread from a per-thread address
    // (threads 0-127: the row's index, clamped to the tile -- GATEUP: its
    // sorted_src entry or, with row tables, its token; DOWN with row tables:
    // its sorted position; the others: their weight-scale entry, clamped to
    // the table), so that no branch makes the weight loads below wait for
    // it.  Without a row index (DOWN over one chunk) threads 0-127 read the
    // tile's first weight-scale entry, whose value they ignore: the
    // weight-scale index tw stays in [0, 2 nb) for every thread, so the
    // address is inside the expert's scale rows.  GATEUP with row tables
    // loads the row's sorted position as well (threads 0-127; the others
    // load their first address again).
    const int ti = min(tid, mc - 1);
    const int tw = tid < kBM ? 0 : min(tid - kBM, 2 * nb - 1);
    const int h = tw / nb, b = tw - h * nb;
    const int64_t wrow = (int64_t)tile.e * (p.N / kBlock) + (GATEUP ? nt : 2 * nt + h);
    const float* sw_src = ((GATEUP && h) ? p.s1 : p.s0) + wrow * nb + b;
    const int32_t* rsrc = GATEUP ? (p.row_tok ? p.row_tok : p.sorted_src) : p.row_pos;
    const uint32_t* src = (tid < kBM && rsrc) ? reinterpret_cast<const uint32_t*>(rsrc + m0 + ti)
                                              : reinterpret_cast<const uint32_t*>(sw_src);
    const uint32_t raw = *src;
    uint32_t raw_pos = 0;
    if (GATEUP) {
      const uint32_t* psrc = (tid < kBM && p.row_pos) ? reinterpret_cast<const uint32_t*>(p.row_pos + m0 + ti) : src;
      raw_pos = *psrc;
    }
#pragma unroll
    for (int s = 0; s < kRing - 1; ++s) MOE_PF_WLOAD(s, s < nb ? s : nb - 1);
    if (tid < kBM) {
      int srow, pos;
      if (GATEUP) {
        srow = p.row_tok ? (int)raw : (int)raw / p.topk;
        pos = p.row_pos ? (int)raw_pos : m0 + tid;
      } else {
        srow = p.row_pos ? (int)raw : m0 + tid;
        pos = srow;
      }
      arow[tid] = (tid < mc && srow >= 0 && srow < p.a_rows) ? srow : -1;
      orow[tid] = pos;
    } else if (tid - kBM < 2 * nb) {
      sw_lds[tid - kBM] = __uint_as_float(raw);
    }
  };

  // acc[j][i]: weight row 8*(i/4) + 4*g2 + i%4 of the operand, expert row 32j + r32.
  v16f acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[j][i] = 0.0f;

  u32x4 ra[2];       // this thread's two 16-byte chunks of one K block of expert rows (ext vectors stay in VGPRs)
  v8i bx[4][2];      // B operands of the step: [expert-row operand][K half]
  v16f dp[2] = {v16f{}, v16f{}};  // operands 2 and 3 of the last step, promoted in the next memory phase
  float sa[4] = {0.0f, 0.0f, 0.0f, 0.0f}, sw0 = 0.0f, sw1 = 0.0f;  // zero: the first memory phase promotes dp (zero) with them

  // The K loop is instantiated for NQ = 1..4 expert-row operands: a tile
  // whose rows fill only NQ of the four 32-row operands (the last tile of
  // an expert) loads, reads and multiplies only those, so a tail tile of
  // 1-32 rows costs its weight stream and a quarter of the MFMAs.  The
  // accumulators of the skipped operands stay 0 and their rows are not
  // written.  NQ is the same in the whole workgroup, so every wave passes
  // the same barriers.
  const int nq = (mc + 31) >> 5;
  auto k_loop = [&](auto nq_tag) {
    constexpr int NQ = decltype(nq_tag)::value;
    constexpr int NA = NQ > 2 ? 2 : 1;  // 16-byte expert-row chunks per thread (chunk 1 holds rows 64-127)
    // Round trip 1: the tile's A row indices (threads 0-127) and the weight
    // scales (the other threads), with the first two weight blocks issued
    // behind them (the row indices are waited for, the weights are not).
    issue_indices_and_weights();
    __syncthreads();
    // Row scales, [K block][row]: element i = m * nb + b of the tile's
    // [row][K block] table goes to sa_lds[b][m] (consecutive threads take
    // consecutive elements, so a wave's loads stay contiguous in memory).
    constexpr int kScalesPerThread = 16;  // covers K <= 8192 in one batch
    const int a_last = arow[mc - 1] >= 0 ? arow[mc - 1] : 0;  // the tile's last row (row 0 if its index is bad)
    // A slot past the table, or on a row without a valid index, holds 0; its
    // load still runs (so that no branch splits the batch) and reads an entry
    // of the tile's own rows instead (a slot past the table: the first row's
    // entry 0; a row without a valid index: the last row's entry).  One
    // stand-in address for all tiles, such as row 0, would be read by every
    // workgroup at once, and one L2 channel would serve them all.
    struct ScaleSlot {
      int m, b, at;
    };
    auto row_scale_slot = [&](int i) {
      const bool in = i < kBM * nb;
      ScaleSlot r;
      r.m = in ? i / nb : 0;
      r.b = in ? i - r.m * nb : 0;
      r.at = in ? r.b * kSaStride + r.m : -1;
      return r;
    };
    auto row_scale_value = [&](const ScaleSlot& sl, int ar) {
      const float v = p.sa[(int64_t)(ar >= 0 ? ar : a_last) * nb + sl.b];
      return (sl.at >= 0 && ar >= 0) ? v : 0.0f;
    };
    // N slots per thread: element i = u * kThreads + tid, whose (m, b)
    // advance by (kThreads / nb, kThreads % nb) per u with a carry instead of
    // a division per element.  `between` runs after the loads are issued and
    // before their values are stored.  Elements beyond 16 slots per thread
    // (K > 8192) follow one at a time.
    auto fill_row_scales = [&](auto n_tag, auto&& between) {
      constexpr int N = decltype(n_tag)::value;
      ScaleSlot ss[N];
      int sar[N];
      float sv[N];
      const int dq = kThreads / nb, dr = kThreads - dq * nb;
      int m = tid / nb, b = tid - m * nb;
  #pragma unroll
      for (int u = 0; u < N; ++u) {
        const bool in = m < kBM;
        ss[u].m = in ? m : 0;
        ss[u].b = in ? b : 0;
        ss[u].at = in ? b * kSaStride + m : -1;
        sar[u] = arow[ss[u].m];
        b += dr;
        m += dq;
        if (b >= nb) {
          b -= nb;
          ++m;
        }
      }
      __builtin_amdgcn_sched_barrier(0);  // all row indices read before the first scale load
  #pragma unroll
      for (int u = 0; u < N; ++u) sv[u] = row_scale_value(ss[u], sar[u]);
      between();
  #pragma unroll
      for (int u = 0; u < N; ++u)
        if (ss[u].at >= 0) sa_lds[ss[u].at] = sv[u];
      for (int i = N * kThreads + tid; i < kBM * nb; i += kThreads) {
        const ScaleSlot sl = row_scale_slot(i);
        sa_lds[sl.at] = row_scale_value(sl, arow[sl.m]);
      }
    };

    // Expert rows: 1024 16-byte chunks per K block, 2 per thread; chunk c
    // covers row c/8, bytes 16*(c%8).  Rows beyond the expert (or with a bad
    // index) load the tile's last row instead (row 0 if that one is bad too):
    // their codes are finite and their scale in sa_lds is 0, so their
    // products promote to exactly 0, and only rows below mc are written.  The
    // stand-in is a row the tile reads anyway, not one address that every
    // tail tile of the launch would read at once.
    const uint8_t* a_src[2];
    int a_dst[2];
  #pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * kThreads;
      const int row = c >> 3, col = (c & 7) * 16;
      const int ar = arow[row];
      a_src[i] = p.a + (int64_t)(ar >= 0 ? ar : a_last) * p.K + col;
      a_dst[i] = swz(row, c & 7);
    }

    const float* swf0 = sw_lds + (GATEUP ? 0 : (wave >> 2)) * nb;  // scale of result rows 0-15
    const float* swf1 = sw_lds + (GATEUP ? 1 : (wave >> 2)) * nb;  // scale of result rows 16-31
    // LDS offsets of this lane's B operand pieces in expert row r32: K chunks
    // 4h + 2 g2 + part; rows 32j + r32 share (row / 2) % 8, hence one offset.
    int bo[2][2];
  #pragma unroll
    for (int h = 0; h < 2; ++h)
  #pragma unroll
      for (int part = 0; part < 2; ++part) bo[h][part] = swz(r32, 4 * h + 2 * g2 + part);

  // Expert rows of K block BLK (clamped to the last block, a harmless
  // reload) into registers, and from there into its LDS stage BLK % 3.
#define MOE_PF_ALOAD(BLK)                                                                  \
  do {                                                                                     \
    const int blk_ = (BLK) < nb ? (BLK) : nb - 1;                                          \
    _Pragma("unroll") for (int i_ = 0; i_ < NA; ++i_)                                      \
      ra[i_] = *reinterpret_cast<const u32x4*>(a_src[i_] + (int64_t)blk_ * kBlock);        \
  } while (0)
#define MOE_PF_ASTORE(BLK)                                                                 \
  do {                                                                                     \
    uint8_t* st_ = smem + ((BLK) % 3) * kHalf;                                             \
    _Pragma("unroll") for (int i_ = 0; i_ < NA; ++i_)                                      \
      *reinterpret_cast<u32x4*>(st_ + a_dst[i_]) = ra[i_];                                 \
  } while (0)
#define MOE_PF_BREAD(J, SB)                                                                \
  do {                                                                                     \
    _Pragma("unroll") for (int h = 0; h < 2; ++h)                                          \
      bx[J][h] = join_v8i(*reinterpret_cast<const uint4*>((SB) + bo[h][0] + (J) * 32 * kLdsRow), \
                          *reinterpret_cast<const uint4*>((SB) + bo[h][1] + (J) * 32 * kLdsRow)); \
  } while (0)
#define MOE_PF_PROMOTE(J, D)                                                               \
  do {                                                                                     \
    const float s0_ = sa[J] * sw0, s1_ = sa[J] * sw1;                                      \
    _Pragma("unroll") for (int i = 0; i < 8; ++i) acc[J][i] += (D)[i] * s0_;               \
    _Pragma("unroll") for (int i = 8; i < 16; ++i) acc[J][i] += (D)[i] * s1_;              \
  } while (0)
  // Each K step j is a memory phase and a compute phase, each ended by a
  // workgroup barrier.  Waves 4-7 run one phase behind waves 0-3 (they pass
  // one extra barrier first), so on every SIMD one wave issues MFMAs while
  // the other issues loads and LDS traffic, instead of both doing the same
  // thing at once.
  // Memory phase of step j: store K block j + 1 (loaded one memory phase
  // earlier) into its stage, load block j + 2 and weight block j + 2, read
  // the step's scales and its first two B operands.  The compute phase reads
  // the other two B operands while the first ones' MFMAs run.
  // Stage safety (three stages, block t in stage t % 3): block j is complete
  // once both halves of the workgroup finished memory phase j - 1, which the
  // lagging half does one phase before the leading half starts memory phase
  // j; its stage is rewritten (block j + 3) in memory phase j + 2, after the
  // lagging half's compute phase j.
#define MOE_PF_MEM(U, J)                                                                   \
  do {                                                                                     \
    const int j_ = (J);                                                                    \
    if (NQ > 2) MOE_PF_PROMOTE(2, dp[0]);                                                  \
    if (NQ > 3) MOE_PF_PROMOTE(3, dp[1]);                                                  \
    MOE_PF_ASTORE(j_ + 1);                                                                 \
    MOE_PF_ALOAD(j_ + 2);                                                                  \
    MOE_PF_WLOAD(((U) + kRing - 1) % kRing, j_ + kRing - 1 < nb ? j_ + kRing - 1 : nb - 1); \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    const uint8_t* sB_ = smem + (j_ % 3) * kHalf;                                          \
    sw0 = swf0[j_];                                                                        \
    sw1 = swf1[j_];                                                                        \
    _Pragma("unroll") for (int q = 0; q < NQ; ++q) sa[q] = sa_lds[j_ * kSaStride + r32 + 32 * q]; \
    MOE_PF_BREAD(0, sB_);                                                                  \
    if (NQ > 1) MOE_PF_BREAD(1, sB_);                                                      \
    __builtin_amdgcn_sched_barrier(0);                                                     \
  } while (0)
  // The two MFMAs of one operand and K block are chained (the second adds
  // onto the first), and a chained MFMA waits for its predecessor to finish;
  // so operands are issued in pairs, each chained MFMA two MFMAs after its
  // predecessor, and a pair is promoted while the next pair runs.
#define MOE_PF_COMP(U, J)                                                                  \
  do {                                                                                     \
    const uint8_t* sB_ = smem + ((J) % 3) * kHalf;                                         \
    v16f d[4];                                                                             \
    _Pragma("unroll") for (int q = 0; q < 4; ++q) d[q] = v16f{};                           \
    d[0] = mfma_f8_32x32x64(wr[U][0], bx[0][0], d[0]);                                     \
    if (NQ > 1) d[1] = mfma_f8_32x32x64(wr[U][0], bx[1][0], d[1]);                         \
    if (NQ > 2) MOE_PF_BREAD(2, sB_);                                                      \
    if (NQ > 3) MOE_PF_BREAD(3, sB_);                                                      \
    d[0] = mfma_f8_32x32x64(wr[U][1], bx[0][1], d[0]);                                     \
    if (NQ > 1) d[1] = mfma_f8_32x32x64(wr[U][1], bx[1][1], d[1]);                         \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    if (NQ > 2) d[2] = mfma_f8_32x32x64(wr[U][0], bx[2][0], d[2]);                         \
    if (NQ > 3) d[3] = mfma_f8_32x32x64(wr[U][0], bx[3][0], d[3]);                         \
    MOE_PF_PROMOTE(0, d[0]);                                                               \
    if (NQ > 2) d[2] = mfma_f8_32x32x64(wr[U][1], bx[2][1], d[2]);                         \
    if (NQ > 3) d[3] = mfma_f8_32x32x64(wr[U][1], bx[3][1], d[3]);                         \
    if (NQ > 1) MOE_PF_PROMOTE(1, d[1]);                                                   \
    __builtin_amdgcn_sched_barrier(0);                                                     \
    if (NQ > 2) dp[0] = d[2];                                                              \
    if (NQ > 3) dp[1] = d[3];                                                              \
    __builtin_amdgcn_sched_barrier(0);                                                     \
  } while (0)
#define MOE_PF_STEP(U, J)                                                                  \
  do {                                                                                     \
    MOE_PF_MEM(U, J);                                                                      \
    __syncthreads();                                                                       \
    MOE_PF_COMP(U, J);                                                                     \
    __syncthreads();                                                                       \
  } while (0)

    // Blocks 0 and 1 of the expert rows and the row scales in one round
    // trip (the first two weight blocks were issued before the previous
    // item's epilogue); block 1 stays in ra for the first memory phase.
    // Row scales in batches sized to the table (4, 8 or 16 slots per
    // thread; every load instruction costs address-unit time, and the down
    // projection's table fills 4 slots); between a batch's loads and its LDS
    // stores go the loads of the first two K blocks of expert rows, so the
    // stores wait for the scales only.
    u32x4 ra0[NA];
    auto issue_blocks = [&]() {
#pragma unroll
      for (int i = 0; i < NA; ++i) ra0[i] = *reinterpret_cast<const u32x4*>(a_src[i]);
      MOE_PF_ALOAD(1);
    };
    const int n_slots = (kBM * nb + kThreads - 1) / kThreads;
    if (n_slots <= 4) fill_row_scales(std::integral_constant<int, 4>{}, issue_blocks);
    else if (n_slots <= 8) fill_row_scales(std::integral_constant<int, 8>{}, issue_blocks);
    else fill_row_scales(std::integral_constant<int, kScalesPerThread>{}, issue_blocks);
#pragma unroll
    for (int i = 0; i < NA; ++i) *reinterpret_cast<u32x4*>(smem + a_dst[i]) = ra0[i];
    __syncthreads();
    if (wave >= 4) __syncthreads();  // the lagging half starts one phase later (wave-uniform branch)

    // kRing = 3 weight slots: three steps per loop iteration keep every slot
    // index static.
    int j0 = 0;
    for (; j0 + kRing <= nb; j0 += kRing) {
      MOE_PF_STEP(0, j0);
      MOE_PF_STEP(1, j0 + 1);
      MOE_PF_STEP(2, j0 + 2);
    }
    if (j0 < nb) MOE_PF_STEP(0, j0);
    if (j0 + 1 < nb) MOE_PF_STEP(1, j0 + 1);
    if (NQ > 2) MOE_PF_PROMOTE(2, dp[0]);
    if (NQ > 3) MOE_PF_PROMOTE(3, dp[1]);
    if (wave < 4) __syncthreads();   // pairs with the lagging half's last barrier
#undef MOE_PF_ALOAD
#undef MOE_PF_ASTORE
#undef MOE_PF_PROMOTE
#undef MOE_PF_BREAD
#undef MOE_PF_MEM
#undef MOE_PF_COMP
#undef MOE_PF_STEP
  };
  switch (nq) {
    case 1: k_loop(std::integral_constant<int, 1>{}); break;
    case 2: k_loop(std::integral_constant<int, 2>{}); break;
    case 3: k_loop(std::integral_constant<int, 3>{}); break;
    default: k_loop(std::integral_constant<int, 4>{}); break;
  }


  if (!GATEUP) {
    // y[m0 + t][nt*256 + 32w + 8*(i/4) + 4*g2 + i%4] for expert row t = 32j + r32.
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = j * 32 + r32;
      if (t < mc) {
        float* dst = p.y + (int64_t)orow[t] * p.N + nt * kBN + wave * 32 + g2 * 4;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<v4f*>(dst + q * 8) = v4f{acc[j][4 * q], acc[j][4 * q + 1], acc[j][4 * q + 2], acc[j][4 * q + 3]};
      }
    }
  } else {

  // GATEUP epilogue: h = SiLU(G) * U for channels 16w + 8*(i/4) + 4*g2 + i%4
  // (i < 8; the up value is acc[j][i + 8]) of rows t = 32j + r32; per-row
  // amax over the lane's 8 channels, the other K-half lane (g2) and the 8
  // waves.
  float hv[4][8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float mx = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      hv[j][i] = silu_mul_fast(acc[j][i], acc[j][i + 8]);
      mx = fmaxf(mx, fabsf(hv[j][i]));
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (g2 == 0) rowmax[wave][j * 32 + r32] = mx;
  }
  __syncthreads();
  uint8_t* qtile = smem;  // [kBM][kLdsRow] swizzled, the K-loop buffers are free now
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int t = j * 32 + r32;
    float amax = rowmax[0][t];
#pragma unroll
    for (int w = 1; w < 8; ++w) amax = fmaxf(amax, rowmax[w][t]);
    const float s = amax / kE4M3Max;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const float* hq = hv[j] + 4 * half;
      const uint32_t packed = quantize4_e4m3(hq[0], hq[1], hq[2], hq[3], s);
      *reinterpret_cast<uint32_t*>(qtile + swz(t, wave) + 8 * half + 4 * g2) = packed;
    }
    if (wave == 0 && g2 == 0 && t < mc) p.sh[(int64_t)orow[t] * (p.N / kBlock) + nt] = s;
  }
  __syncthreads();
  // 128 rows x 128 bytes = 1024 16-byte chunks, 2 per thread.
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = tid + i * kThreads;
    const int row = c >> 3, col = (c & 7) * 16;
    if (row < mc)
      *reinterpret_cast<uint4*>(p.qh + (int64_t)orow[row] * p.N + nt * kBlock + col) =
          *reinterpret_cast<const uint4*>(qtile + swz(row, c & 7));
  }
  }  // GATEUP epilogue
#undef MOE_PF_WLOAD
}

template <bool GATEUP>
moe_status_t launch_prefill(const PrefillArgs& a, int64_t max_mtiles, hipStream_t stream) {
  int64_t grid = max_mtiles * a.n_tiles;
  grid = (grid + kXcd - 1) / kXcd * kXcd;
  if (grid > 0x7fffffff) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: grid too large");
  if ((int64_t)a.N * a.K > 0x7fffffff)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: one expert matrix (%d x %d) exceeds 2 GiB", a.N, a.K);
  const size_t lds = (size_t)kStages * kHalf + sizeof(float) * ((size_t)kSaStride + 2) * (a.K / kBlock);
  if (lds > 150 * 1024) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: K=%d needs %zu bytes of LDS", a.K, lds);
  const hipError_t ae = hipFuncSetAttribute(reinterpret_cast<const void*>(&ffn_prefill_kernel<GATEUP>),
                                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (ae != hipSuccess) return fail(MOE_ERR_HIP, "ffn_prefill: LDS attribute: %s", hipGetErrorString(ae));
  MOE_LAUNCH(GATEUP ? "ffn_prefill_gateup" : "ffn_prefill_down", (ffn_prefill_kernel<GATEUP>), dim3((unsigned)grid), dim3(kThreads), lds, stream, a);
  return check_launch(GATEUP ? "ffn_prefill_gateup" : "ffn_prefill_down");
}

}  // namespace

// Shapes the prefill kernels take (checked before anything is enqueued).
moe_status_t prefill_shape_check(const moe_dims_t& d) {
  if (d.hidden % kBN) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "prefill regime needs H %% 256 == 0 (H=%d)", d.hidden);
  if ((int64_t)d.inter * d.hidden > 0x7fffffff)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: one expert matrix (%d x %d) exceeds 2 GiB", d.inter,
                d.hidden);
  const int kmax = d.hidden > d.inter ? d.hidden : d.inter;
  // The [2][K/128] weight-scale table is loaded one entry per thread, by the threads after the first 128.
  if (2 * (kmax / kBlock) > kThreads - kBM)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: K=%d exceeds %d", kmax, (kThreads - kBM) / 2 * kBlock);
  const size_t lds = (size_t)kStages * kHalf + sizeof(float) * ((size_t)kSaStride + 2) * (kmax / kBlock);
  if (lds > 150 * 1024) return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: K=%d needs %zu bytes of LDS", kmax, lds);
  return MOE_OK;
}

// Bound on the 128-row m-tiles of R routed rows over E experts.
int64_t prefill_max_mtiles(int64_t R, int64_t E) { return (R + kBM - 1) / kBM + (R < E ? R : E); }

// The tiles workspace of a launch over n_units experts: the index tables,
// the m-tile descriptors [max_mtiles] and, for a launch over several chunks
// (table_rows > 0), the row tables [table_rows] each.
size_t prefill_tiles_bytes(int64_t n_units, int64_t max_mtiles, int64_t table_rows) {
  const size_t tab = ((size_t)table_rows * sizeof(int32_t) + 15) & ~(size_t)15;
  return tiles_desc_offset(n_units) + (size_t)max_mtiles * sizeof(int4) + 2 * tab;
}

size_t prefill_tile_workspace(const moe_dims_t& d, int32_t T) {
  return prefill_tiles_bytes(d.n_experts, prefill_max_mtiles((int64_t)T * d.topk, d.n_experts), 0);
}

// Gate/up then down over the expert-sorted rows that r describes (the
// experts' rows of one chunk, or of several chunks each sorted on its own;
// see prefill_tiles_kernel).  The weight stacks hold the r.n_units experts;
// qx/sx hold r.tokens rows, sorted_src, qh/sh and y_rows r.rows rows (chunk
// c's from row c * r.chunk_rows).  tiles: prefill_tiles_bytes(r.n_units,
// r.max_mtiles, r.n_chunks > 1 ? r.rows : 0) bytes, 16-byte aligned.
moe_status_t run_ffn_prefill_view(const moe_dims_t& d, const PrefillRows& r, const uint8_t* qx, const float* sx,
                                  const int32_t* sorted_src, const uint8_t* w_gate, const float* s_gate,
                                  const uint8_t* w_up, const float* s_up, const uint8_t* w_down, const float* s_down,
                                  float* y_rows, uint8_t* qh, float* sh, int32_t* tiles, hipStream_t stream) {
  moe_status_t st0 = prefill_shape_check(d);
  if (st0 != MOE_OK) return st0;
  if (r.rows > 0x7fffffff || r.n_units < 1 || r.n_chunks < 1 || (int64_t)r.n_chunks * r.n_units > 0x7fffffff)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: %lld rows, %d experts x %d chunks", (long long)r.rows,
                r.n_units, r.n_chunks);
  if (r.n_chunks > 65535 || r.n_units > 65535)
    return fail(MOE_ERR_UNSUPPORTED_SHAPE, "ffn_prefill: %d chunks x %d experts", r.n_chunks, r.n_units);
  uint8_t* tb = reinterpret_cast<uint8_t*>(tiles);
  int32_t* vstart = reinterpret_cast<int32_t*>(tb + tiles_index_bytes(r.n_units));
  int4* desc = reinterpret_cast<int4*>(tb + tiles_desc_offset(r.n_units));
  int32_t* row_pos = nullptr;
  int32_t* row_tok = nullptr;
  MOE_LAUNCH("prefill_tiles", prefill_tiles_kernel, dim3(1), dim3(1024), 0, stream, r.offsets, r.off_stride,
             r.n_units, r.n_chunks, tiles, vstart, desc, r.max_mtiles);
  moe_status_t st = check_launch("prefill_tiles");
  if (st != MOE_OK) return st;
  if (r.n_chunks > 1) {
    row_pos = reinterpret_cast<int32_t*>(reinterpret_cast<uint8_t*>(desc) + (size_t)r.max_mtiles * sizeof(int4));
    row_tok = row_pos + ((r.rows + 3) & ~(int64_t)3);
    MOE_LAUNCH("prefill_rows", prefill_rows_kernel, dim3((unsigned)r.n_chunks, (unsigned)r.n_units), dim3(256), 0,
               stream, r.offsets, r.off_stride, r.chunk_rows, r.chunk_tokens, sorted_src, d.topk, vstart, row_pos,
               row_tok);
    st = check_launch("prefill_rows");
    if (st != MOE_OK) return st;
  }

  PrefillArgs g{};
  g.a = qx; g.sa = sx; g.sorted_src = sorted_src; g.row_pos = row_pos; g.row_tok = row_tok;
  g.topk = d.topk; g.a_rows = r.tokens;
  g.mtile_start = tiles; g.desc = desc; g.max_mtiles = r.max_mtiles; g.n_units = r.n_units;
  g.w0 = w_gate; g.s0 = s_gate; g.w1 = w_up; g.s1 = s_up;
  g.N = d.inter; g.K = d.hidden; g.n_tiles = d.inter / kBlock;
  g.qh = qh; g.sh = sh; g.y = nullptr;
  st = launch_prefill<true>(g, r.max_mtiles, stream);
  if (st != MOE_OK) return st;

  PrefillArgs dn{};
  dn.a = qh; dn.sa = sh; dn.sorted_src = nullptr; dn.row_pos = row_pos; dn.row_tok = nullptr;
  dn.topk = d.topk; dn.a_rows = (int)r.rows;
  dn.mtile_start = tiles; dn.desc = desc; dn.max_mtiles = r.max_mtiles; dn.n_units = r.n_units;
  dn.w0 = w_down; dn.s0 = s_down; dn.w1 = nullptr; dn.s1 = nullptr;
  dn.N = d.hidden; dn.K = d.inter; dn.n_tiles = d.hidden / kBN;
  dn.y = y_rows; dn.qh = nullptr; dn.sh = nullptr;
  return launch_prefill<false>(dn, r.max_mtiles, stream);
}

moe_status_t run_ffn_prefill(const moe_dims_t& d, int32_t T, const uint8_t* qx, const float* sx,
                             const int32_t* offsets, const int32_t* sorted_src, const uint8_t* w_gate,
                             const float* s_gate, const uint8_t* w_up, const float* s_up, const uint8_t* w_down,
                             const float* s_down, float* y_rows, uint8_t* qh, float* sh, int32_t* tiles,
                             hipStream_t stream) {
  PrefillRows r{};
  r.offsets = offsets; r.off_stride = 0; r.n_units = d.n_experts; r.n_chunks = 1; r.chunk_rows = 0;
  r.chunk_tokens = 0; r.tokens = T; r.rows = (int64_t)T * d.topk;
  r.max_mtiles = prefill_max_mtiles(r.rows, d.n_experts);
  return run_ffn_prefill_view(d, r, qx, sx, sorted_src, w_gate, s_gate, w_up, s_up, w_down, s_down, y_rows, qh, sh,
                              tiles, stream);
}

}  // namespace moe
