// kernels.h -- launch interface of the gfx950 kernels of libmoesplit
// (internal to the library; the public C ABI is include/moesplit.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

namespace msk {

constexpr int kChunkUnits = 64;    // FFN intermediate units per chunk
constexpr int kMaxTasks = 200;     // tasks passed by value in one FFN launch (3.3 KiB of kernel arguments)
static_assert(kMaxTasks <= 256, "find_task_of reads at most 256 task starts");
constexpr int kFfnLanesPerUnit = 8;  // lanes sharing one unit row in phase 1
constexpr int kMaxExperts = 512;   // grouping / ranking kernels' LDS bound
constexpr int kMaxTopK = 64;
constexpr int kMaxModelDim = 8192;  // d_model limit of every kernel
// Work-groups per chunk the FFN kernel supports at this width and element
// size: 16-byte loads, and a one-row tile's down-projection accumulators
// (column passes x elements per load) within 32 registers, i.e. at most 4
// column passes in bf16 and 8 in fp32.
inline int max_ffn_splits(int d, int elem) {
  int subs = 4;
  while (subs > 1 && d > (64 / subs) * kFfnLanesPerUnit * (16 / elem) * (2 * elem)) subs >>= 1;
  return subs;
}

enum Dtype { kF32 = 0, kBF16 = 1 };

// Router logits in the fixed fp32 order, for one or two router weights
// (the layer's own, and the next layer's for the speculative prediction):
// logits[t][e] = h_t . w[:, e] (+ bias[e]).
struct LogitsArgs {
  const void* h;          // [T][d] model dtype
  int T, d, E;
  int dtype;
  const void* wr;         // [d][E] model dtype (NULL: this router is absent)
  const void* wt;         // the same router transposed, [E][d] (read by the kernels)
  const float* bias;      // [E] or NULL
  float* logits;          // [T][E]
  const void* wr2;        // second router or NULL
  const void* wt2;
  const float* bias2;
  float* logits2;
};

// Routing of T >= kManyTokens tokens runs over many work-groups: logits in
// tiles of 8 tokens x 16 experts per wave, selection and per-block expert
// counts for blocks of route_block_tokens(T, K) tokens, one work-group for the
// scans over blocks (and the prediction ranking), then the scatter of the
// grouping.  Fewer tokens: one wave per router row against a block of up to
// four staged token rows (or one wave per logit when such a block does not
// fit LDS), then one work-group for everything after the logits.
constexpr int kManyTokens = 64;
// Tokens per block: 4 (one per wave of the selection), or 16 from
// kBigBlockTokens tokens on (with at most 16 selected experts per token), so
// that the scan over blocks stays short (measured: Qwen3-shaped routing of
// 2048 tokens with the prediction router 124 -> 106 us; at 64 and 512 tokens
// 16-token blocks were slower).
constexpr int kBigBlockTokens = 1024;
inline int route_block_tokens(int T, int K) { return (T >= kBigBlockTokens && K <= 16) ? 16 : 4; }
// Blocks of any token count up to max_T.
inline int route_block_cap(int max_T, int K) {
  const int small = (std::min(max_T, kBigBlockTokens - 1) + 3) / 4;
  return std::max(small, (max_T + route_block_tokens(max_T, K) - 1) / route_block_tokens(max_T, K));
}


// One work-group: top-K selection with lowest-index ties and Eq. (2) gate
// weights, the stable token-to-expert grouping, and the ranking of the
// prediction scores (summed softmax of the second logits).
struct RouteArgs {
  int T, E, K;
  int renormalize;
  const float* logits;      // [T][E] or NULL: no selection / grouping
  int32_t* idx;             // [T][K]
  float* w;                 // [T][K]
  int32_t* offsets;         // [E+1]
  int32_t* perm;            // [T*K] slot at each grouped position
  int32_t* pos;             // [T*K] grouped position of each slot
  int32_t* host_offsets;    // [E+1] host-visible copy (mapped) or NULL
  const float* logits_pred; // [T][E] or NULL: no ranking
  float* score;             // [E]
  int32_t* order;           // [E]
  float* host_score;        // host-visible or NULL
  int32_t* host_order;      // host-visible or NULL
  // host-visible completion word or NULL: set to seq once every host-visible
  // output above is visible to the host (the host polls it instead of
  // waiting for the launch to complete)
  int32_t* host_seq;
  int32_t seq;
  // many-token workspace (ignored below kManyTokens tokens)
  int32_t* lrank;           // [T*K] rank of a slot among its block's slots of the same expert
  int32_t* blk;             // [E][nblk_cap] per-block expert counts, then their prefix sums
  float* psc;               // [E][nblk_cap] per-block prediction score sums (a block's expert-major, so
                            // that the sums over blocks read contiguous memory)
  int32_t nblk_cap;
};
// Logits launch, then the route launch on them.
hipError_t launch_logits_route(const LogitsArgs& a, const RouteArgs& ra, hipStream_t s);

// One FFN task: chunks [chunk_lo, chunk_lo + n_chunks) of one expert whose
// chunk c lives at base + c * chunk_bytes.  expert >= 0: routed expert (its
// tokens come from the grouping); expert = -1 - s: shared expert s (all T
// tokens).  wg_begin: first work-group of the task in the launch grid.
struct FfnTask {
  const unsigned char* base;
  int32_t expert;
  int32_t chunk_lo;
  int32_t n_chunks;
  int32_t wg_begin;
};

// The kernels' copy of a task (16 bytes, so that one launch holds many):
// chunk_lo < 65536 and expert in int16 range, checked at launch.
struct FfnTaskK {
  const unsigned char* base;
  int32_t wg_begin;
  int16_t expert;
  uint16_t chunk_lo;
  FfnTaskK() = default;
  FfnTaskK(const FfnTask& t)
      : base(t.base), wg_begin(t.wg_begin), expert(static_cast<int16_t>(t.expert)),
        chunk_lo(static_cast<uint16_t>(t.chunk_lo)) {}
};

// Each chunk is computed by `subs` work-groups of 64 / subs units each; the
// work-group for (chunk c, sub s) writes partial plane c * subs + s.
struct FfnArgs {
  const void* h;              // [T][d] model dtype
  const int32_t* offsets;     // [E+1] grouping
  const int32_t* perm;        // [TK]
  float* part;                // routed partials [rows_routed][n_planes][d]
  float* part_sh;             // shared partials [n_shared][rows_shared][n_planes_sh][d]
  uint64_t chunk_bytes;       // bytes of one chunk (3 * 64 * d * elem)
  int64_t sh_plane;           // floats per shared expert in part_sh
  int32_t rows_routed;        // row stride of one routed chunk plane (max T*K)
  int32_t rows_shared;        // row stride of one shared chunk plane (max T)
  int32_t d, K, T;
  int32_t dtype;
  int32_t n_tasks;
  int32_t n_wg;               // total work-groups: sum of task chunks * subs
  int32_t subs;               // work-groups per chunk: 1, 2 or 4
  int32_t n_planes;           // routed partial planes: n_chunks * subs
  int32_t n_planes_sh;        // shared partial planes: n_chunks_sh * subs
  int32_t bits;               // 0: chunks in the model dtype; 2 or 4: b-bit codes
                              // (bf16 activations, routed experts, subs = 1)
  FfnTaskK tasks[kMaxTasks];  // ascending wg_begin
};
static_assert(sizeof(FfnTaskK) == 16, "task records are 16 bytes");
static_assert(sizeof(FfnArgs) <= 3400, "FFN kernel arguments within the size other launches use");
// Launches n_wg work-groups; max_tok must be at least the token count of
// every task (tokens past the launch's tiles are not computed).
hipError_t launch_ffn(const FfnArgs& a, int max_tok, hipStream_t s);

// Chunks of b-bit experts (FfnArgs::bits = 2 or 4): affine codes with one
// fp16 scale s and zero z per group of 64 elements along each matrix's input
// axis, w = (q - z) * s.  Per 64-unit chunk:
//   Gq, Uq [64 units][d / 64 groups][8 b bytes]; Dq [d columns][8 b bytes]
//   (the chunk's 64 units of one down column form one group);
//   Gm, Um [64 units][d / 64] and Dm [d] words: fp16 scale | fp16 zero << 16.
// Inside a group, 32-bit word m holds the codes of elements 2p and 2p + 1,
// p = m * 16 / b + j, at bits j * b and 16 + j * b (j < 16 / b).
inline uint64_t q_chunk_bytes(int d, int bits) {
  return 3ull * kChunkUnits * d * bits / 8 + 12ull * d;
}
inline uint64_t q_off_uq(int d, int bits) { return 1ull * kChunkUnits * d * bits / 8; }
inline uint64_t q_off_dq(int d, int bits) { return 2ull * kChunkUnits * d * bits / 8; }
inline uint64_t q_off_gm(int d, int bits) { return 3ull * kChunkUnits * d * bits / 8; }
inline uint64_t q_off_um(int d, int bits) { return q_off_gm(d, bits) + 4ull * d; }
inline uint64_t q_off_dm(int d, int bits) { return q_off_gm(d, bits) + 8ull * d; }
// Quantized chunks need d a multiple of 64 in [256, 8192].
inline bool q_supported(int d) { return d % 64 == 0 && d >= 256 && d <= kMaxModelDim; }

// Prefill (many tokens per expert) runs on the matrix cores in two steps:
//  gate/up (mma_gateup): act[row][f] = bf16(silu(h_row . G_f) * (h_row . U_f))
//    for a task's chunk range, 64 rows x 64 / gu_split units per work-group
//    (m_tiles * n_chunks * gu_split work-groups per task); runs per segment
//    as data lands (disjoint columns of act);
//  down (mma_down): out[row][:] = sum_f act[row][f] * D_f over all of the
//    expert's chunks (chunks < split at base, the rest at base2), 64 rows x
//    256 columns per work-group, written as the single partial plane.
constexpr int kMaxMmaTasks = 192;  // tasks by value in one matrix-core launch (7.7 KiB of kernel arguments)
static_assert(kMaxMmaTasks <= 256, "find_task_of reads at most 256 task starts");
// gate/up work-groups per chunk and row tile: 4 (16 units each) for launches
// of fewer than kGuSplitBelow row-tile chunks, else 1 (whole chunks)
constexpr int kGuSplitBelow = 256;
constexpr int kMmaRows = 64;     // rows (token slots) per work-group
constexpr int kGdMaxRows = 192;  // rows per tile of the LDS-staged gate/up kernel (bf16, d % 128 == 0)
// chunks per work-group of the LDS-staged gate/up kernel: four for a task of
// at most 64 rows and at least 16 chunks (its activation rows then feed four
// chunks' weights, and it still spreads over enough work-groups), else two
// (measured: DeepSeek-V2-Lite prefill 512, 22 chunks per expert, gate/up 184
// -> 175 us; Qwen3 prefill 2048, 12 chunks, 215 -> 223 us with four)
__host__ __device__ inline int gd_group_chunks(int task_rows, int task_chunks) {
  return task_rows <= 64 && task_chunks >= 16 ? 4 : 2;
}
constexpr int kMmaCols = 256;    // output columns per down work-group

struct MmaTask {
  const unsigned char* base;   // chunk c at base + c * chunk_bytes
  const unsigned char* base2;  // down: chunks >= split at base2 + c * chunk_bytes
  int32_t expert;              // >= 0 routed expert; -1 - s shared expert s
  int32_t chunk_lo;            // gate/up: first chunk
  int32_t n_chunks;            // gate/up: chunks in the task; down: all chunks
  int32_t split;               // down: first chunk read from base2
  int32_t wg_begin;
  int32_t m_tiles;             // row tiles of this task
};

struct MmaArgs {
  const void* h;               // [T][d] bf16
  const int32_t* offsets;      // [E+1]
  const int32_t* perm;         // [TK]
  uint16_t* act;               // routed [rows_routed][f_pad] bf16
  uint16_t* act_sh;            // shared [n_shared][rows_shared][f_pad_sh] bf16
  float* part;                 // down output, routed [rows_routed][d] (one plane)
  float* part_sh;              // shared [n_shared] planes of sh_plane floats
  uint64_t chunk_bytes;
  int64_t sh_plane;
  int32_t d, K, T;
  int32_t f_pad, f_pad_sh;     // act row strides (chunks * 64)
  int32_t rows_shared;         // shared rows per expert (max T)
  int32_t n_tasks, n_wg;
  int32_t ncb;                 // down: column blocks (ceil(d / kMmaCols))
  int32_t gu_split;            // gate/up: work-groups per chunk and row tile (1 or 4; 1 for b-bit chunks)
  int32_t bits;                // 0: bf16 chunks; 2 or 4: b-bit chunks (q_chunk_bytes layout)
  int32_t ksplit;              // down, b-bit: chunk ranges per (row tile, column block), each summed
                               // into its own partial plane [row][ksplit][d]; 1 for bf16
  int32_t tile_rows;           // rows per row tile: kMmaRows, or kGdMaxRows for the bf16 gate/up of
                               // whole chunks (gu_split 1, d % 128 == 0)
  // tasks planned on the device (launch_prefill_plan), or null for `tasks`:
  // dtasks[dcount[0]] over dcount[1] work-groups; the grid is an upper bound
  // and work-groups past dcount[1] exit (LDS-staged kernels only)
  const MmaTask* dtasks;
  const int32_t* dcount;
  MmaTask tasks[kMaxMmaTasks];
};
// kernel arguments of this size were measured to reach the kernels intact
static_assert(sizeof(MmaArgs) <= 8000, "matrix-core kernel arguments within 8000 bytes");
hipError_t launch_mma_gateup(const MmaArgs& a, hipStream_t s);
hipError_t launch_mma_down(const MmaArgs& a, hipStream_t s);

// Prefill work planned on the device right after the routing, so that the
// resident experts' matrix-core launches need no host round trip: for every
// routed expert with tokens and resident chunks, a gate/up task over those
// chunks, and a down task when all of its chunks are resident; for every
// shared expert, both.  Row tiles of tile_rows rows; tasks in expert order,
// then the shared experts.  One work-group of kMaxPlanTasks threads.
constexpr int kMaxPlanTasks = 256;   // routed + shared experts of a planned forward
constexpr int kMaxPlanShared = 4;
struct PlanArgs {
  const int32_t* offsets;            // [E+1] grouping offsets of this forward
  MmaTask* gu;                       // [kMaxPlanTasks] out
  MmaTask* dn;                       // [kMaxPlanTasks] out
  int32_t* counts;                   // [4] out: gate/up tasks and work-groups, down tasks and work-groups
  const unsigned char* cache_base;   // top of routed expert e at cache_base + top_bytes * slot[e]
  uint64_t top_bytes;
  const unsigned char* shared[kMaxPlanShared];
  int32_t E, T, n_chunks, n_chunks_sh, n_sh, ncb, tile_rows;
  int16_t res[kMaxPlanTasks];        // resident chunks of routed expert e (a snapshot at launch)
  int16_t slot[kMaxPlanTasks];       // its cache slot (when res[e] > 0)
};
hipError_t launch_prefill_plan(const PlanArgs& a, hipStream_t s);

// Host-to-device copy of `bytes` (a multiple of 16; both addresses 16-byte
// aligned) from pinned host memory that the device can address (src is its
// device-side address) into device memory, by a streaming kernel of
// kH2dWorkGroups work-groups of kH2dThreads threads.  Unlike a DMA-engine
// copy, it orders after other streams' work through ordinary kernel-to-
// kernel dependencies.
//
// Reads of host memory stay in flight for microseconds, and a work-group
// that shares a CU with them waits behind them: an HBM-bound FFN launch
// beside a copy ran 2.8x slower than alone while their work-groups could
// share CUs, 1.2x while they could not.  So each copy work-group holds all
// of its CU's LDS (kCuLdsBytes), which keeps every work-group that requests
// LDS off that CU, and kernels that need no LDS request kGuardLds bytes at
// launch for the same reason.
constexpr int kH2dWorkGroups = 16;
constexpr int kH2dThreads = 512;
constexpr unsigned kCuLdsBytes = 160 * 1024;  // LDS of one gfx950 CU
constexpr unsigned kGuardLds = 64;
hipError_t launch_h2d(void* dst, const void* src, uint64_t bytes, hipStream_t s);
// A streaming kernel for a device-to-device copy (no LDS held), over enough
// work-groups to run at HBM rate.
constexpr int kD2dWorkGroups = 1024;
hipError_t launch_d2d(void* dst, const void* src, uint64_t bytes, hipStream_t s);

// Glue between stacked layers: out[t] = x / sqrt(mean(x^2) + eps) with
// x = h[t] + y[t], in fp32, stored in the model dtype (bf16: round to
// nearest even).  One work-group per token.
hipError_t launch_residual_norm(const void* h, const float* y, void* out, int T, int d, int dtype, float eps,
                                hipStream_t s);

// y[t] = sum_k w[t][k] * sum_c part[c][pos[t*K+k]] + sum_s sum_c part_sh[s][c][t],
// c over the partial planes (chunks * subs), in two launches: a first pass
// over plane groups into `red`, then the weighted sum per token.
struct CombineArgs {
  const float* part;
  const float* part_sh;
  const int32_t* pos;         // [T*K]
  const float* w;             // [T*K]
  float* y;                   // [T][d]
  float* red;                 // [pg][T*(K+n_shared)][d] first-pass sums
  int64_t sh_plane;
  int32_t rows_routed, rows_shared;
  int32_t n_planes, n_planes_sh, n_shared;
  int32_t T, K, d;
  int32_t pg;                 // plane groups of the first pass (combine_groups)
};
// Plane groups for the first pass at this shape (a power of two <= 16).
int combine_groups(int T, int K, int n_shared, int d, int n_planes);
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);

}  // namespace msk
