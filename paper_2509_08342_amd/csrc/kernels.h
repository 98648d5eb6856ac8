// kernels.h -- launch interface of the gfx950 kernels of libmoesplit
// (internal to the library; the public C ABI is include/moesplit.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace msk {

constexpr int kChunkUnits = 64;    // FFN intermediate units per chunk
constexpr int kMaxTasks = 120;     // tasks passed by value in one FFN launch
constexpr int kFfnThreads = 512;   // threads per FFN work-group (8 waves)
constexpr int kMaxExperts = 512;   // grouping / ranking kernels' LDS bound
constexpr int kMaxTopK = 64;

enum Dtype { kF32 = 0, kBF16 = 1 };

// Router: logits in the fixed fp32 order, top-K with lowest-index ties,
// softmax weights; optionally the next layer's softmax probabilities.
struct RouterArgs {
  const void* h;          // [T][d] model dtype
  int T, d, E, K;
  int dtype;
  int renormalize;
  const void* wr;         // [d][E] model dtype (NULL: no selection)
  const float* bias;      // [E] or NULL
  int32_t* idx;           // [T][K]
  float* w;               // [T][K]
  const void* wr_next;    // [d][E] (NULL: no prediction)
  const float* bias_next; // [E] or NULL
  float* p_pred;          // [T][E] next-layer probabilities
};
hipError_t launch_router(const RouterArgs& a, hipStream_t s);

// Grouping of the T*K (token, k) slots by expert (stable counting sort).
struct GroupArgs {
  const int32_t* idx;     // [TK]
  int TK, E;
  int32_t* offsets;       // [E+1]
  int32_t* perm;          // [TK] slot at each grouped position
  int32_t* pos;           // [TK] grouped position of each slot
  int32_t* host_offsets;  // [E+1] host-visible copy (pinned, mapped) or NULL
};
hipError_t launch_group(const GroupArgs& a, hipStream_t s);

// Prediction ranking: score[e] = sum_t p_pred[t][e]; order by descending
// score, lower index first on ties.
struct RankArgs {
  const float* p_pred;    // [T][E]
  int T, E;
  float* score;           // [E] device
  int32_t* order;         // [E] device
  float* host_score;      // [E] host-visible or NULL
  int32_t* host_order;    // [E] host-visible or NULL
};
hipError_t launch_rank(const RankArgs& a, hipStream_t s);

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

struct FfnArgs {
  const void* h;              // [T][d] model dtype
  const int32_t* offsets;     // [E+1] grouping
  const int32_t* perm;        // [TK]
  float* part;                // routed partials [n_chunks][rows_routed][d]
  float* part_sh;             // shared partials [n_shared][n_chunks_sh][rows_shared][d]
  uint64_t chunk_bytes;       // bytes of one chunk (3 * 64 * d * elem)
  int64_t sh_plane;           // floats per shared expert in part_sh
  int32_t rows_routed;        // row stride of one routed chunk plane (max T*K)
  int32_t rows_shared;        // row stride of one shared chunk plane (max T)
  int32_t d, K, T;
  int32_t dtype;
  int32_t n_tasks;
  int32_t n_wg;               // total work-groups
  FfnTask tasks[kMaxTasks];
};
// Launches ceil(n_wg) work-groups; max_tok bounds the tokens of any task.
hipError_t launch_ffn(const FfnArgs& a, int max_tok, hipStream_t s);

// y[t] = sum_k w[t][k] * sum_c part[c][pos[t*K+k]] + sum_s sum_c part_sh[s][c][t].
struct CombineArgs {
  const float* part;
  const float* part_sh;
  const int32_t* pos;         // [T*K]
  const float* w;             // [T*K]
  float* y;                   // [T][d]
  int64_t sh_plane;
  int32_t rows_routed, rows_shared;
  int32_t n_chunks, n_chunks_sh, n_shared;
  int32_t T, K, d;
};
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);

}  // namespace msk
