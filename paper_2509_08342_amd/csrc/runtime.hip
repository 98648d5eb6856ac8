// runtime.hip -- host runtime of libmoesplit: context, device-pool carve-up,
// pinned chunk-packed expert store, per-layer top-segment caches, staging
// buffer with chunk-group copies, prefetch queue, and the per-layer forward
// that overlaps resident-segment compute with the transfer of missing
// segments (arXiv 2509.08342, Sec. 3.1-3.2, Eq. (5)-(6)).
//
// Streams: the caller's compute stream runs routing, grouping, the resident
// FFN launch and the combine; the library's copy stream carries every H2D
// segment transfer; the library's side stream computes streamed chunk groups
// as their copy events fire.  All streams have the default priority.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <functional>
#include <mutex>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <deque>
#include <string>
#include <thread>
#include <vector>

#include "kernels.h"
#include "moesplit.h"
#include "planner.h"

namespace {
// Per-forward work buffers of ms_forward_noalloc, for callers that cannot
// allocate: a fixed array in device memory, one copy per GPU, held until the
// process ends.
constexpr uint64_t kStaticScratchBytes = 64ull << 20;
constexpr int kMaxDevices = 64;
}  // namespace

// In host code the name is only a stand-in for the symbol: each GPU's copy
// is reached through the device address hipGetSymbolAddress returns for it
// (scratch_address below), never through the name.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

constexpr int kUnits = msk::kChunkUnits;
constexpr uint64_t kAlign = 256;
// H2D copy granularity: prefetch copies are speculative -- when the routing
// arrives, queued groups are dropped but the groups in flight complete, used
// or not -- so they go in small groups, 1/16 of an expert within
// [4 MiB, 16 MiB]; a miss is needed whole, so its copies go in large groups
// (each copy launch leaves a gap of ~12 us on the link).  Measured on the
// decode layers, stacks and decoders of the Mixtral (bf16 and 2-bit),
// DeepSeek and Qwen3 shapes: 2-bit Mixtral (55 MB experts) gains 6-10% per
// token from 4 MiB prefetch groups over 16 MiB, bf16 Mixtral (352 MB) is
// within 1% from 4 to 16 MiB.
constexpr uint64_t kGroupMinBytes = 4ull << 20;

constexpr uint64_t kGroupMaxBytes = 16ull << 20;
constexpr uint64_t kMissGroupTargetBytes = 64ull << 20;
constexpr int kPrefetchWindow = 2;                   // prefetch groups in flight
constexpr int kMaxD = msk::kMaxModelDim;
constexpr int kReserved = 1 << 30;                   // BufSlot::use_order of a reserved slot
constexpr int kRouteCheckMs = 20;  // the host's wait for a routing checks the stream this often

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

struct Shape {
  int L, d, F, E, K, n_sh, F_sh, dtype, renorm, max_T, n_buf, subs;
  int elem;
  int bits;  // 0: routed experts in the model dtype; 2 or 4: b-bit codes
  uint64_t chunk_bytes;
  int n_chunks, n_chunks_sh;
  uint64_t expert_bytes, shared_bytes;
  int group_chunks;       // chunks per H2D copy group of a prefetch
  int miss_group_chunks;  // ... of a miss
  // fixed pool layout (byte offsets)
  uint64_t off_router, off_bias, off_shared, off_logits, off_logits2, off_offsets, off_perm, off_pos;
  uint64_t off_part, off_part_sh, off_red, off_act, off_act_sh, off_score, off_order, off_buffer, fixed_bytes;
  uint64_t off_router_t, off_lrank, off_blk, off_psc;
  uint64_t off_plan;  // prefill tasks planned on the device: gate/up, down, counts
  int nblk_cap;  // token blocks of the many-token routing
  int down_splits;  // prefill down projection of b-bit chunks: chunk ranges (partial planes) per slot
  uint64_t router_stride, bias_stride, part_bytes, part_sh_bytes;
  int64_t sh_plane;
};

ms_status derive_shape(const ms_model_desc* d, Shape* s, std::string* err) {
  if (!d) {
    *err = "desc is NULL";
    return MS_E_INVALID;
  }
  if (d->n_layers <= 0 || d->d_model <= 0 || d->d_ff <= 0 || d->n_experts <= 0 || d->top_k <= 0 ||
      d->top_k > d->n_experts || d->n_shared < 0 || d->max_tokens <= 0 || d->n_buffer_slots < 0 ||
      (d->dtype != MS_F32 && d->dtype != MS_BF16) || (d->n_shared > 0 && d->d_ff_shared <= 0) ||
      (d->ffn_splits != 0 && d->ffn_splits != 1 && d->ffn_splits != 2 && d->ffn_splits != 4)) {
    *err = "invalid model description";
    return MS_E_INVALID;
  }
  // the prefill kernels stage activation slabs of 128 and the decode
  // kernels' tiles assume a few 64-wide k pieces: d_model in [256, 8192]
  if (d->d_model % 64 != 0 || d->d_model < 256 || d->d_model > kMaxD) {
    *err = "d_model must be a multiple of 64 in [256, 8192]";
    return MS_E_UNSUPPORTED;
  }
  if (d->n_experts > msk::kMaxExperts || d->top_k > msk::kMaxTopK) {
    *err = "n_experts <= 512 and top_k <= 64 are supported";
    return MS_E_UNSUPPORTED;
  }
  if (static_cast<int64_t>(d->max_tokens) * d->top_k > (1 << 24)) {
    *err = "max_tokens * top_k too large";
    return MS_E_UNSUPPORTED;
  }
  // the FFN kernels' task records hold chunk indices in 16 bits and expert
  // ids (-1 - s for shared expert s) in int16
  if (d->d_ff > 65535 * 64 || (d->n_shared > 0 && d->d_ff_shared > 65535 * 64) || d->n_shared > 32767) {
    *err = "d_ff and d_ff_shared must be at most 4194240, n_shared at most 32767";
    return MS_E_UNSUPPORTED;
  }
  s->L = d->n_layers;
  s->d = d->d_model;
  s->F = d->d_ff;
  s->E = d->n_experts;
  s->K = d->top_k;
  s->n_sh = d->n_shared;
  s->F_sh = d->n_shared > 0 ? d->d_ff_shared : 0;
  s->dtype = d->dtype;
  s->renorm = d->renormalize ? 1 : 0;
  s->max_T = d->max_tokens;
  s->n_buf = d->n_buffer_slots > 0 ? d->n_buffer_slots : 2 * d->top_k;
  s->elem = d->dtype == MS_BF16 ? 2 : 4;
  s->bits = d->expert_bits;
  if (s->bits != 0) {
    if (s->bits != 2 && s->bits != 4) {
      *err = "expert_bits must be 0, 2 or 4";
      return MS_E_INVALID;
    }
    if (d->dtype != MS_BF16 || d->n_shared != 0 || d->d_ff % kUnits != 0 || !msk::q_supported(d->d_model) ||
        d->ffn_splits > 1) {
      *err = "b-bit experts need bf16 activations, no shared experts, d_ff a multiple of 64, "
             "d_model a multiple of 64 in [256, 8192] and one work-group per chunk";
      return MS_E_UNSUPPORTED;
    }
  }
  s->chunk_bytes = s->bits ? msk::q_chunk_bytes(s->d, s->bits) : 3ull * kUnits * s->d * s->elem;
  s->n_chunks = (s->F + kUnits - 1) / kUnits;
  s->n_chunks_sh = (s->F_sh + kUnits - 1) / kUnits;
  // b-bit prefill down projection: a work-group per (64 rows, 256 columns)
  // loops over the expert's chunks; ranges of >= 16 chunks (at most 8)
  // spread a launch for one expert over more work-groups
  s->down_splits = s->bits ? std::max(1, std::min(8, s->n_chunks / 16)) : 1;
  s->expert_bytes = s->chunk_bytes * s->n_chunks;
  s->shared_bytes = s->chunk_bytes * s->n_chunks_sh;
  const uint64_t group_bytes = std::min(kGroupMaxBytes, std::max(kGroupMinBytes, s->expert_bytes / 16));
  s->group_chunks = static_cast<int>(std::max<uint64_t>(1, group_bytes / s->chunk_bytes));
  s->miss_group_chunks = static_cast<int>(std::max<uint64_t>(1, kMissGroupTargetBytes / s->chunk_bytes));
  // work-groups per chunk: one for experts of many chunks (each work-group
  // then streams more bytes, and fewer partial planes reach the combine),
  // two otherwise, doubled until the experts a forward can activate give
  // the FFN kernel >= 256 work-groups (measured best on this GPU for the
  // Mixtral-, DeepSeek- and Qwen3-shaped decode layers)
  const int max_subs = msk::max_ffn_splits(d->d_model, d->dtype == MS_BF16 ? 2 : 4);
  if (d->ffn_splits > max_subs) {
    *err = "ffn_splits too large for this d_model and dtype";
    return MS_E_UNSUPPORTED;
  }
  if (s->bits != 0) {
    s->subs = 1;  // the b-bit kernel takes a whole chunk per work-group
  } else if (d->ffn_splits > 0) {
    s->subs = d->ffn_splits;
  } else {
    const int64_t active = std::min<int64_t>(s->E, static_cast<int64_t>(s->max_T) * s->K) + s->n_sh;
    const int64_t work = active * s->n_chunks;
    s->subs = std::min(max_subs, s->n_chunks >= 128 ? 1 : 2);
    while (s->subs < max_subs && work * s->subs < 256) s->subs *= 2;
  }

  const uint64_t TK = static_cast<uint64_t>(s->max_T) * s->K;
  uint64_t off = 0;
  s->router_stride = align_up(static_cast<uint64_t>(s->d) * s->E * s->elem, kAlign);
  s->off_router = off;
  off += s->router_stride * s->L;
  s->off_router_t = off;  // the same routers transposed, [E][d]
  off += s->router_stride * s->L;
  s->bias_stride = align_up(static_cast<uint64_t>(s->E) * 4, kAlign);
  s->off_bias = off;
  off += s->bias_stride * s->L;
  s->off_shared = off;
  off += align_up(s->shared_bytes, kAlign) * s->n_sh * s->L;
  s->off_logits = off;
  off += align_up(static_cast<uint64_t>(s->max_T) * s->E * 4, kAlign);
  s->off_logits2 = off;
  off += align_up(static_cast<uint64_t>(s->max_T) * s->E * 4, kAlign);
  s->off_offsets = off;
  off += align_up(static_cast<uint64_t>(s->E + 1) * 4, kAlign);
  s->off_perm = off;
  off += align_up(TK * 4, kAlign);
  s->off_pos = off;
  off += align_up(TK * 4, kAlign);
  s->part_bytes = static_cast<uint64_t>(s->n_chunks) * s->subs * TK * s->d * 4;
  s->off_part = off;
  off += align_up(s->part_bytes, kAlign);
  s->sh_plane = static_cast<int64_t>(s->n_chunks_sh) * s->subs * s->max_T * s->d;
  s->part_sh_bytes = static_cast<uint64_t>(s->sh_plane) * 4 * s->n_sh;
  s->off_part_sh = off;
  off += align_up(s->part_sh_bytes, kAlign);
  // first-pass combine sums [pg][T*(K+n_shared)][d]: with one plane group
  // that is the slots of max_T tokens; with more, pg * slots * ceil(d/256)
  // stays <= 1024 (combine_groups)
  const uint64_t red_bytes = std::max<uint64_t>(static_cast<uint64_t>(s->max_T) * (s->K + s->n_sh),
                                                512 / ((s->d + 255) / 256)) * s->d * 4;
  s->off_red = off;
  off += align_up(red_bytes, kAlign);
  // prefill path (bf16): SwiGLU activations [rows][chunks * 64] per routed
  // slot and per shared expert and token
  s->off_act = off;
  s->off_act_sh = off;
  if (s->dtype == MS_BF16) {
    off += align_up(TK * s->n_chunks * kUnits * 2, kAlign);
    s->off_act_sh = off;
    off += align_up(static_cast<uint64_t>(s->n_sh) * s->max_T * s->n_chunks_sh * kUnits * 2, kAlign);
  }

  // many-token routing workspace
  s->nblk_cap = msk::route_block_cap(s->max_T, s->K);
  s->off_lrank = off;
  off += align_up(TK * 4, kAlign);
  s->off_blk = off;
  off += align_up(static_cast<uint64_t>(s->E) * s->nblk_cap * 4, kAlign);
  s->off_psc = off;
  off += align_up(static_cast<uint64_t>(s->E) * s->nblk_cap * 4, kAlign);

  s->off_plan = off;
  off += align_up(2 * msk::kMaxPlanTasks * sizeof(msk::MmaTask) + 4 * sizeof(int32_t), kAlign);

  s->off_score = off;
  off += align_up(static_cast<uint64_t>(s->E) * 4, kAlign);
  s->off_order = off;
  off += align_up(static_cast<uint64_t>(s->E) * 4, kAlign);
  s->off_buffer = off;
  off += s->expert_bytes * s->n_buf;  // expert_bytes is a multiple of 256
  s->fixed_bytes = off;
  return MS_OK;
}

int top_units_for(float r, int F) {
  double x = static_cast<double>(r) * F / kUnits + 0.5;
  int units = static_cast<int>(x) * kUnits;
  return std::max(0, std::min(units, F));
}

// Pack one SwiGLU FFN (w_gate, w_up [d][F], w_down [F][d]) into chunk order:
// per 64-unit chunk, the gate block, the up block and the down block.  Gate
// and up blocks are k-tiled -- unit u's weights for k in [64 kb, 64 kb + 64)
// form one 64-element piece at ((kb * 64) + u) * 64 -- and the down block
// holds the 64 down rows, each d-contiguous.  Units past F are zero.
template <typename T>
void pack_expert_t(const T* wg, const T* wu, const T* wd, int d, int F, int n_chunks, T* dst) {
  constexpr int KT = 64;
  auto work = [&](int c0, int c1) {
    for (int c = c0; c < c1; ++c) {
      T* G = dst + static_cast<size_t>(c) * 3 * kUnits * d;
      T* U = G + static_cast<size_t>(kUnits) * d;
      T* D = U + static_cast<size_t>(kUnits) * d;
      const int f0 = c * kUnits;
      const int nu = std::min(kUnits, F - f0);
      if (nu < kUnits) std::memset(G, 0, sizeof(T) * 3 * kUnits * d);
      for (int j = 0; j < d; ++j) {
        const T* gr = wg + static_cast<size_t>(j) * F + f0;
        const T* ur = wu + static_cast<size_t>(j) * F + f0;
        const size_t base = static_cast<size_t>(j / KT) * kUnits * KT + (j % KT);
        for (int u = 0; u < nu; ++u) {
          G[base + static_cast<size_t>(u) * KT] = gr[u];
          U[base + static_cast<size_t>(u) * KT] = ur[u];
        }
      }
      for (int u = 0; u < nu; ++u)
        std::memcpy(D + static_cast<size_t>(u) * d, wd + static_cast<size_t>(f0 + u) * d, sizeof(T) * d);
    }
  };
  const int n_threads = std::max(1, std::min<int>(16, static_cast<int>(std::thread::hardware_concurrency())));
  if (n_chunks < 4 || n_threads == 1) {
    work(0, n_chunks);
    return;
  }
  std::vector<std::thread> th;
  const int per = (n_chunks + n_threads - 1) / n_threads;
  for (int i = 0; i < n_threads; ++i) {
    const int c0 = i * per, c1 = std::min(n_chunks, c0 + per);
    if (c0 < c1) th.emplace_back(work, c0, c1);
  }
  for (auto& t : th) t.join();
}

void pack_expert(const void* wg, const void* wu, const void* wd, int d, int F, int n_chunks, int elem,
                 void* dst) {
  if (elem == 2)
    pack_expert_t(static_cast<const uint16_t*>(wg), static_cast<const uint16_t*>(wu),
                  static_cast<const uint16_t*>(wd), d, F, n_chunks, static_cast<uint16_t*>(dst));
  else
    pack_expert_t(static_cast<const float*>(wg), static_cast<const float*>(wu),
                  static_cast<const float*>(wd), d, F, n_chunks, static_cast<float*>(dst));
}

// Pack one b-bit expert (gate_q, up_q [F][d b/8] and down_q [d][F b/8]
// codes, element i of a row at bits (i % (8/b)) b of byte i / (8/b); meta
// [rows][in/64][2] fp16 (scale, zero)) into the chunk order of the b-bit
// kernel: per chunk Gq, Uq, Dq, Gm, Um, Dm (msk::q_chunk_bytes), each
// group's 64 codes as 2b words of code pairs (elements 2p, 2p + 1 at bits
// j b and 16 + j b of word p / (16 / b), j = p % (16 / b)).
void pack_group_pairs(const uint8_t* row, int first, int bits, uint32_t* out) {
  const int per = 8 / bits, ppw = 16 / bits, words = 2 * bits;
  const unsigned mask = (1u << bits) - 1u;
  auto code = [&](int i) { return (static_cast<unsigned>(row[(first + i) / per]) >> (((first + i) % per) * bits)) & mask; };
  for (int m = 0; m < words; ++m) {
    uint32_t w = 0;
    for (int j = 0; j < ppw; ++j) {
      const int p = m * ppw + j;
      w |= code(2 * p) << (j * bits);
      w |= code(2 * p + 1) << (16 + j * bits);
    }
    out[m] = w;
  }
}

void pack_expert_q(const uint8_t* gq, const uint16_t* gm, const uint8_t* uq, const uint16_t* um, const uint8_t* dq,
                   const uint16_t* dm, int d, int F, int bits, uint8_t* dst) {
  const int n_chunks = F / kUnits, ngr = d / 64, ngr_f = F / 64;
  const size_t qrow_in = static_cast<size_t>(d) * bits / 8;   // bytes of one gate/up code row
  const size_t drow_in = static_cast<size_t>(F) * bits / 8;   // bytes of one down code row
  const size_t gbytes = 8ull * bits;                          // bytes of one group's codes
  const uint64_t cb = msk::q_chunk_bytes(d, bits);
  auto work = [&](int c0, int c1) {
    for (int c = c0; c < c1; ++c) {
      uint8_t* base = dst + cb * c;
      uint32_t* Gq = reinterpret_cast<uint32_t*>(base);
      uint32_t* Uq = reinterpret_cast<uint32_t*>(base + msk::q_off_uq(d, bits));
      uint32_t* Dq = reinterpret_cast<uint32_t*>(base + msk::q_off_dq(d, bits));
      uint32_t* Gm = reinterpret_cast<uint32_t*>(base + msk::q_off_gm(d, bits));
      uint32_t* Um = reinterpret_cast<uint32_t*>(base + msk::q_off_um(d, bits));
      uint32_t* Dm = reinterpret_cast<uint32_t*>(base + msk::q_off_dm(d, bits));
      for (int u = 0; u < kUnits; ++u) {
        const size_t f = static_cast<size_t>(c) * kUnits + u;
        for (int g = 0; g < ngr; ++g) {
          const size_t grp = static_cast<size_t>(u) * ngr + g;
          pack_group_pairs(gq + f * qrow_in, g * 64, bits, Gq + grp * gbytes / 4);
          pack_group_pairs(uq + f * qrow_in, g * 64, bits, Uq + grp * gbytes / 4);
          Gm[grp] = gm[(f * ngr + g) * 2] | static_cast<uint32_t>(gm[(f * ngr + g) * 2 + 1]) << 16;
          Um[grp] = um[(f * ngr + g) * 2] | static_cast<uint32_t>(um[(f * ngr + g) * 2 + 1]) << 16;
        }
      }
      for (int col = 0; col < d; ++col) {
        pack_group_pairs(dq + static_cast<size_t>(col) * drow_in, c * kUnits, bits, Dq + col * gbytes / 4);
        const size_t mi = (static_cast<size_t>(col) * ngr_f + c) * 2;
        Dm[col] = dm[mi] | static_cast<uint32_t>(dm[mi + 1]) << 16;
      }
    }
  };
  const int n_threads = std::max(1, std::min<int>(16, static_cast<int>(std::thread::hardware_concurrency())));
  if (n_chunks < 4 || n_threads == 1) {
    work(0, n_chunks);
    return;
  }
  std::vector<std::thread> th;
  const int per = (n_chunks + n_threads - 1) / n_threads;
  for (int i = 0; i < n_threads; ++i) {
    const int c0 = i * per, c1 = std::min(n_chunks, c0 + per);
    if (c0 < c1) th.emplace_back(work, c0, c1);
  }
  for (auto& t : th) t.join();
}

struct Group {
  int c_lo = 0, c_hi = 0;
  bool issued = false;
  bool prefetch = false;  // issued by prefetch
  bool used = false;      // consumed by a forward
  bool pre = false;       // computed by the running forward's resident launch
  bool landed = false;    // its copy was seen complete (not polled again)
};

struct BufSlot {
  unsigned char* base = nullptr;  // device, expert_bytes
  int layer = -1, expert = -1;
  int first_chunk = 0;            // content covers chunks [first_chunk, n_chunks)
  std::vector<Group> groups;
  std::vector<hipEvent_t> gev;    // per group copy-done event
  hipEvent_t last_read = nullptr; // side-stream event after the last reader
  bool has_last_read = false;
  uint64_t tick = 0;              // last use
  int use_order = -1;             // order of use in the running forward (-1: not used,
                                  // kReserved: holds an expert not yet processed)
};

struct LayerState {
  bool router_set = false, bias_set = false;
  std::vector<int> blob_of;        // [E] -> index into ctx blobs, -1 unset
  std::vector<bool> shared_set;
  // cache configuration (Sec. 3.4)
  bool configured = false;
  uint64_t budget = 0;
  float r = 0.f;
  int top_units = 0, top_chunks = 0;
  uint64_t top_bytes = 0;
  int slots = 0;                   // C_i
  unsigned char* cache_base = nullptr;
  std::vector<int> slot_of;        // [E] -> cache slot or -1
  std::vector<int> slot_owner;     // [C_i] -> expert or -1
  std::vector<hipEvent_t> pending_loads;
  hipEvent_t last_fwd = nullptr;
  bool has_last_fwd = false;
  // the end of this layer's last forward is recorded into last_fwd only when
  // something waits for it (a marker between two kernels costs the stream a
  // few microseconds); until then it is the end of fwd_stream's work so far
  bool fwd_unrecorded = false;
  hipStream_t fwd_stream = nullptr;
  // prediction made for this layer (Eq. (3)), checked at its next routing
  std::vector<int> pred_order;
  bool has_pred = false;
  ms_layer_stats st{};
  // cache priority state (Eq. (4)) and the configurator's statistics
  // (Sec. 3.4.2): activations by priority rank, by prediction rank, and the
  // priority rank of each prediction rank
  std::vector<double> mu, nu;        // [E]
  std::vector<uint64_t> last_use;    // [E] forward count at the last activation (0: never)
  uint64_t clock = 0;                // forwards of this layer
  uint64_t q = 0, q_pred = 0;        // tokens; tokens of forwards with a prediction
  std::vector<uint64_t> hit_hist, pred_act, pred_rank;  // [E], [E], [E][E]
};

struct TlRec {
  int kind, layer;
  uint64_t bytes;
  hipEvent_t e0, e1;
};

struct PendingGroup {
  int slot, group;
};

}  // namespace

struct ms_ctx {
  Shape s{};
  std::string err;
  bool poisoned = false;
  // online cache replacement (Sec. 3.3) and the priority's parameters
  bool side_work = false;  // the running forward enqueued kernels on the side stream
  bool side2_work = false;  // ... on the second side stream
  int policy = MS_CACHE_STATIC;
  double rho = 0.25, omega = 128.0;
  uint64_t rng = 0x9e3779b97f4a7c15ull;
  int device = 0;
  unsigned char* scratch_addr = nullptr;  // this device's copy of `scratch`
  unsigned char* pool = nullptr;
  uint64_t pool_bytes = 0;
  hipStream_t copy = nullptr, side = nullptr;
  hipStream_t side2 = nullptr;  // prefill: every other missing expert's compute
  // host-to-device copies: the copy kernel, or (MS_COPY_DMA) the DMA
  // engines except while the copy stream waits on unfinished work of
  // another stream (copy_waits)
  int copy_engine = MS_COPY_KERNEL;
  bool dma_warm = false;  // a DMA transfer has completed in this context
  std::vector<hipEvent_t> copy_waits;
  // pinned host store
  std::vector<unsigned char*> blobs;      // pinned, coherent host memory (never cached by the GPU)
  std::vector<unsigned char*> blobs_dev;  // the same memory's device-side addresses
  int blob_cap = 0;  // 0: unlimited
  // host-visible small buffers written by kernels
  int32_t* h_offsets = nullptr;
  int32_t* h_order = nullptr;
  float* h_score = nullptr;
  int32_t* d_offsets_map = nullptr;  // device views of the three buffers above
  int32_t* d_order_map = nullptr;
  float* d_score_map = nullptr;
  // routing completion word (host-visible): the routing launch of a forward
  // sets it to that forward's number once the offsets are visible
  int32_t* h_seq = nullptr;
  int32_t* d_seq_map = nullptr;
  uint32_t route_seq = 0;
  std::vector<LayerState> layers;
  std::vector<BufSlot> buf;
  uint64_t tick = 0;
  std::deque<PendingGroup> pf_queue;
  std::vector<PendingGroup> pf_inflight;
  hipEvent_t ev_route = nullptr, ev_res = nullptr, ev_side_done = nullptr, ev_last = nullptr;
  hipEvent_t ev_side2_done = nullptr;
  bool has_last = false;
  // the most recent end-of-work record: ev_last (prediction) or the layer's
  // last_fwd (a forward records only that one; each marker between kernels
  // costs the stream a few microseconds)
  hipEvent_t last_ev = nullptr;
  hipStream_t last_stream = nullptr;
  std::vector<hipEvent_t> free_events;
  // timeline
  bool tl_on = false;
  int tl_cap = 0;
  hipEvent_t tl_origin = nullptr;
  std::vector<TlRec> tl;
  std::vector<hipEvent_t> tl_pool;

  // ms_forward_noalloc: while set, the per-forward work buffers (the pool
  // range [off_logits, off_buffer)) live at work_base instead
  unsigned char* work_base = nullptr;

  unsigned char* dev(uint64_t off) {
    if (work_base && off >= s.off_logits && off < s.off_buffer) return work_base + (off - s.off_logits);
    return pool + off;
  }
};

namespace {

#define MS_HIP(call)                                                                  \
  do {                                                                                \
    hipError_t e_ = (call);                                                           \
    if (e_ != hipSuccess) return poison(ctx, #call, e_);                              \
  } while (0)

ms_status poison(ms_ctx* ctx, const char* what, hipError_t e) {
  ctx->poisoned = true;
  ctx->err = std::string("HIP error in ") + what + ": " + hipGetErrorString(e);
  return MS_E_HIP;
}

// Device address of the current GPU's copy of `scratch`, looked up once per
// device (ms_create calls this with the context's device current).
std::mutex g_scratch_mu;
unsigned char* g_scratch_addr[kMaxDevices] = {};

hipError_t scratch_address(int device, unsigned char** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipSuccess;
  if (!g_scratch_addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[device] = static_cast<unsigned char*>(p);
  }
  *out = g_scratch_addr[device];
  return hipSuccess;
}

ms_status fail(ms_ctx* ctx, ms_status st, const std::string& msg) {
  ctx->err = msg;
  return st;
}

#define MS_CHECK_CTX(ctx)                                   \
  do {                                                      \
    if (!(ctx)) return MS_E_INVALID;                        \
    if ((ctx)->poisoned) return MS_E_HIP;                   \
  } while (0)

hipError_t new_event(ms_ctx* ctx, hipEvent_t* ev) {
  if (!ctx->free_events.empty()) {
    *ev = ctx->free_events.back();
    ctx->free_events.pop_back();
    return hipSuccess;
  }
  return hipEventCreateWithFlags(ev, hipEventDisableTiming);
}

// ---- timeline

int tl_begin(ms_ctx* ctx, hipStream_t st, int kind, int layer, uint64_t bytes) {
  if (!ctx->tl_on || static_cast<int>(ctx->tl.size()) >= ctx->tl_cap) return -1;
  TlRec r{kind, layer, bytes, nullptr, nullptr};
  for (hipEvent_t* e : {&r.e0, &r.e1}) {
    if (!ctx->tl_pool.empty()) {
      *e = ctx->tl_pool.back();
      ctx->tl_pool.pop_back();
    } else if (hipEventCreate(e) != hipSuccess) {
      return -1;
    }
  }
  if (hipEventRecord(r.e0, st) != hipSuccess) return -1;
  ctx->tl.push_back(r);
  return static_cast<int>(ctx->tl.size()) - 1;
}

void tl_end(ms_ctx* ctx, int idx, hipStream_t st) {
  if (idx < 0) return;
  (void)hipEventRecord(ctx->tl[idx].e1, st);
}

// ---- copies

// Order the copy stream after `ev`, recorded on another stream.  Finished
// work needs no wait.  Unfinished work gets a stream wait, and until it has
// finished the copies use the copy kernel: a DMA transfer queued behind such
// a wait can hold the host inside the runtime's copy call for the length of
// the awaited work.
ms_status copy_after(ms_ctx* ctx, hipEvent_t ev) {
  const hipError_t q = hipEventQuery(ev);
  if (q == hipSuccess) return MS_OK;
  if (q != hipErrorNotReady) MS_HIP(q);
  MS_HIP(hipStreamWaitEvent(ctx->copy, ev, 0));
  ctx->copy_waits.push_back(ev);
  return MS_OK;
}

// Whether some wait queued by copy_after is still unfinished (an event
// recorded again since then only reports later work, so the answer errs
// towards the copy kernel).
bool copy_waits_pending(ms_ctx* ctx) {
  auto& w = ctx->copy_waits;
  w.erase(std::remove_if(w.begin(), w.end(), [](hipEvent_t e) { return hipEventQuery(e) == hipSuccess; }), w.end());
  return !w.empty();
}

// H2D copy on the copy stream from a host blob (src: its host address,
// src_dev: its device-side address), by the streaming copy kernel, or in
// MS_COPY_DMA mode by the DMA engines when nothing unfinished is awaited.
ms_status issue_copy(ms_ctx* ctx, void* dst, const void* src, const void* src_dev, uint64_t bytes, int kind,
                     int layer) {
  const int ti = tl_begin(ctx, ctx->copy, kind, layer, bytes);
  if (ctx->copy_engine == MS_COPY_DMA && !copy_waits_pending(ctx))
    MS_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, ctx->copy));
  else
    MS_HIP(msk::launch_h2d(dst, src_dev, bytes, ctx->copy));
  tl_end(ctx, ti, ctx->copy);
  return MS_OK;
}

// Issue one group of a staging slot on the copy stream and record its event.
ms_status issue_group(ms_ctx* ctx, int si, int gi, bool prefetch) {
  BufSlot& b = ctx->buf[si];
  Group& g = b.groups[gi];
  const uint64_t cb = ctx->s.chunk_bytes;
  const int bi = ctx->layers[b.layer].blob_of[b.expert];
  const uint64_t off = cb * g.c_lo, bytes = cb * (g.c_hi - g.c_lo);
  ms_status st = issue_copy(ctx, b.base + off, ctx->blobs[bi] + off, ctx->blobs_dev[bi] + off, bytes,
                            prefetch ? MS_IV_COPY_PREFETCH : MS_IV_COPY_MISS, b.layer);
  if (st != MS_OK) return st;
  MS_HIP(hipEventRecord(b.gev[gi], ctx->copy));
  g.issued = true;
  g.prefetch = prefetch;
  LayerState& L = ctx->layers[b.layer];
  if (prefetch)
    L.st.bytes_prefetch += bytes;
  else
    L.st.bytes_miss += bytes;
  return MS_OK;
}

// Whether group gi of slot si has landed: its event is polled until it has
// been seen complete once (each poll is a runtime call on the host).
hipError_t group_landed(ms_ctx* ctx, int si, int gi) {
  Group& g = ctx->buf[si].groups[gi];
  if (g.landed) return hipSuccess;
  if (!g.issued) return hipErrorNotReady;
  const hipError_t q = hipEventQuery(ctx->buf[si].gev[gi]);
  if (q == hipSuccess) g.landed = true;
  return q;
}

// Point a staging slot at (layer, e) covering chunks [first, n_chunks).  The
// copy stream first waits for the slot's previous readers.
ms_status assign_slot(ms_ctx* ctx, int si, int layer, int e, int first, bool miss) {
  BufSlot& b = ctx->buf[si];
  if (b.has_last_read) {
    const ms_status st = copy_after(ctx, b.last_read);
    if (st != MS_OK) return st;
  }
  b.layer = layer;
  b.expert = e;
  b.first_chunk = first;
  b.groups.clear();
  // at most (miss_)group_chunks per copy, in groups of near-equal size (a
  // small tail copy runs far below the link rate)
  const int n = ctx->s.n_chunks, G = miss ? ctx->s.miss_group_chunks : ctx->s.group_chunks;
  const int ng = (n - first + G - 1) / G;
  const int per = ng > 0 ? (n - first + ng - 1) / ng : 1;
  for (int c = first; c < n; c += per) {
    Group g;
    g.c_lo = c;
    g.c_hi = std::min(n, c + per);
    b.groups.push_back(g);
  }
  if (b.gev.size() < b.groups.size()) return fail(ctx, MS_E_STATE, "staging slot has fewer copy events than groups");
  return MS_OK;
}

// Resident chunks of expert e in layer L: [0, top_chunks) if its top is
// cached, none otherwise.
int resident_chunks(const LayerState& L, int e) { return L.slot_of[e] >= 0 ? L.top_chunks : 0; }

void clear_slot(BufSlot& b) {
  b.layer = -1;
  b.expert = -1;
  b.groups.clear();
}

int find_slot(ms_ctx* ctx, int layer, int e) {
  for (int i = 0; i < static_cast<int>(ctx->buf.size()); ++i)
    if (ctx->buf[i].layer == layer && ctx->buf[i].expert == e) return i;
  return -1;
}

// Pick a staging slot for new content.  Prefers empty slots, then the least
// recently used slot not used by the running forward; if allow_busy, falls
// back to the slot whose readers in the running forward were enqueued first
// (the copy stream will wait for them).  Reserved slots are never taken;
// returns -1 if nothing can be taken.
int pick_victim(ms_ctx* ctx, bool allow_busy) {
  int best = -1;
  for (int i = 0; i < static_cast<int>(ctx->buf.size()); ++i) {
    const BufSlot& b = ctx->buf[i];
    if (b.use_order >= 0) continue;
    if (b.layer < 0) return i;
    if (best < 0 || b.tick < ctx->buf[best].tick) best = i;
  }
  if (best >= 0 || !allow_busy) return best;
  for (int i = 0; i < static_cast<int>(ctx->buf.size()); ++i) {
    const int u = ctx->buf[i].use_order;
    if (u >= kReserved) continue;
    if (best < 0 || u < ctx->buf[best].use_order) best = i;
  }
  return best;
}

// Active experts of a forward that miss chunks, in processing order: those
// whose missing part a staging slot already holds come first, so that their
// reserved slots are released before any other miss needs a victim.
std::vector<int> miss_order(ms_ctx* ctx, int layer, const std::vector<int32_t>& offs,
                            const std::vector<char>* skip) {
  const LayerState& L = ctx->layers[layer];
  std::vector<int> first, rest;
  for (int e = 0; e < ctx->s.E; ++e) {
    if (offs[e + 1] == offs[e] || resident_chunks(L, e) >= ctx->s.n_chunks) continue;
    if (skip && (*skip)[e]) continue;
    const int si = find_slot(ctx, layer, e);
    if (si >= 0 && ctx->buf[si].first_chunk <= resident_chunks(L, e))
      first.push_back(e);
    else
      rest.push_back(e);
  }
  first.insert(first.end(), rest.begin(), rest.end());
  return first;
}

// Keep up to kPrefetchWindow prefetch groups in flight.
ms_status pump_prefetch(ms_ctx* ctx) {
  for (size_t i = 0; i < ctx->pf_inflight.size();) {
    const PendingGroup pg = ctx->pf_inflight[i];
    const hipError_t q = group_landed(ctx, pg.slot, pg.group);
    if (q == hipSuccess) {
      ctx->pf_inflight.erase(ctx->pf_inflight.begin() + i);
    } else if (q == hipErrorNotReady) {
      ++i;
    } else {
      return poison(ctx, "hipEventQuery(prefetch)", q);
    }
  }
  while (static_cast<int>(ctx->pf_inflight.size()) < kPrefetchWindow && !ctx->pf_queue.empty()) {
    const PendingGroup pg = ctx->pf_queue.front();
    ctx->pf_queue.pop_front();
    ms_status st = issue_group(ctx, pg.slot, pg.group, true);
    if (st != MS_OK) return st;
    ctx->pf_inflight.push_back(pg);
  }
  return MS_OK;
}

// Drop every prefetch group not yet issued (Sec. 3.2: the prefetch stops when
// a layer's routing result arrives).  Slots left with nothing issued become
// empty.
void terminate_prefetch(ms_ctx* ctx) {
  for (const PendingGroup& pg : ctx->pf_queue) {
    BufSlot& b = ctx->buf[pg.slot];
    const Group& g = b.groups[pg.group];
    if (b.layer >= 0)
      ctx->layers[b.layer].st.bytes_prefetch_dropped += ctx->s.chunk_bytes * (g.c_hi - g.c_lo);
  }
  ctx->pf_queue.clear();
  for (BufSlot& b : ctx->buf) {
    if (b.layer < 0) continue;
    bool any = false;
    for (const Group& g : b.groups) any = any || g.issued;
    if (!any) clear_slot(b);
  }
}


// Enqueue the prefetch of experts[0..n) of `layer` (in order) into free
// staging slots: the bottom if the top is cached, else the whole expert.
ms_status enqueue_prefetch(ms_ctx* ctx, int layer, const int32_t* experts, int n) {
  LayerState& L = ctx->layers[layer];
  const int nch = ctx->s.n_chunks;
  for (int i = 0; i < n; ++i) {
    const int e = experts[i];
    const int res = resident_chunks(L, e);
    if (res >= nch) continue;                       // already whole in VRAM
    if (L.blob_of[e] < 0) continue;                 // weights not set
    const int have = find_slot(ctx, layer, e);
    if (have >= 0 && ctx->buf[have].first_chunk <= res) {
      // already (partly) buffered: queue what has not been issued
      BufSlot& hb = ctx->buf[have];
      bool queued = false;
      for (const PendingGroup& pg : ctx->pf_queue) queued = queued || pg.slot == have;
      if (queued) continue;
      for (int gi = 0; gi < static_cast<int>(hb.groups.size()); ++gi)
        if (!hb.groups[gi].issued && hb.groups[gi].c_hi > res) ctx->pf_queue.push_back({have, gi});
      hb.tick = ++ctx->tick;
      continue;
    }
    int si = have >= 0 ? have : pick_victim(ctx, false);
    if (si < 0) break;                              // no free slot left
    if (ctx->buf[si].use_order >= 0) break;
    // a slot already queued for prefetch must not be taken over
    bool queued = false;
    for (const PendingGroup& pg : ctx->pf_queue) queued = queued || pg.slot == si;
    for (const PendingGroup& pg : ctx->pf_inflight) queued = queued || pg.slot == si;
    if (queued) break;
    ms_status st = assign_slot(ctx, si, layer, e, res, false);
    if (st != MS_OK) return st;
    ctx->buf[si].tick = ++ctx->tick;
    for (int gi = 0; gi < static_cast<int>(ctx->buf[si].groups.size()); ++gi)
      ctx->pf_queue.push_back({si, gi});
  }
  return pump_prefetch(ctx);
}

ms_status check_layer(ms_ctx* ctx, int layer) {
  if (layer < 0 || layer >= ctx->s.L) return fail(ctx, MS_E_INVALID, "layer out of range");
  return MS_OK;
}

// ---- cache priority (Eq. (4)) and configurator statistics (Sec. 3.4.2)

double lcp_priority(const ms_ctx* ctx, const LayerState& L, int e) {
  return L.mu[e] * std::pow(ctx->rho, L.nu[e] / ctx->omega);
}

// Experts in descending order of `key`, ties to the lower index.
std::vector<int> order_by(const std::vector<double>& key) {
  std::vector<int> o(key.size());
  for (size_t i = 0; i < o.size(); ++i) o[i] = static_cast<int>(i);
  std::stable_sort(o.begin(), o.end(), [&](int a, int b) { return key[a] > key[b]; });
  return o;
}

std::vector<int> priority_order(const ms_ctx* ctx, const LayerState& L) {
  std::vector<double> p(ctx->s.E);
  for (int e = 0; e < ctx->s.E; ++e) p[e] = lcp_priority(ctx, L, e);
  return order_by(p);
}

// One forward's routing (tokens per expert from the grouping offsets) into
// the statistics, ranked by the priorities before this forward, then the
// priority state.  A batch is one step of the activation interval.
void update_plan_stats(ms_ctx* ctx, LayerState& L, const std::vector<int32_t>& offs, int T) {
  const int E = ctx->s.E;
  const std::vector<int> order = priority_order(ctx, L);
  std::vector<int> rank(E);
  for (int r = 0; r < E; ++r) rank[order[r]] = r;
  for (int e = 0; e < E; ++e) L.hit_hist[rank[e]] += static_cast<uint64_t>(offs[e + 1] - offs[e]);
  if (L.has_pred && static_cast<int>(L.pred_order.size()) == E) {
    for (int y = 0; y < E; ++y) {
      const int e = L.pred_order[y];
      L.pred_act[y] += static_cast<uint64_t>(offs[e + 1] - offs[e]);
      L.pred_rank[static_cast<size_t>(y) * E + rank[e]] += static_cast<uint64_t>(T);
    }
    L.q_pred += static_cast<uint64_t>(T);
  }
  L.q += static_cast<uint64_t>(T);
  L.clock += 1;
  for (int e = 0; e < E; ++e) {
    const int n = offs[e + 1] - offs[e];
    L.mu[e] += n;
    L.nu[e] = n > 0 ? 0.0 : L.nu[e] + 1.0;
    if (n > 0) L.last_use[e] = L.clock;
  }
}

uint64_t next_random(ms_ctx* ctx) {  // splitmix64
  uint64_t z = (ctx->rng += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

// The replacement policy's ranking key of each expert (larger = keep).
std::vector<double> policy_key(ms_ctx* ctx, const LayerState& L) {
  const int E = ctx->s.E;
  std::vector<double> k(E);
  for (int e = 0; e < E; ++e) {
    switch (ctx->policy) {
      case MS_CACHE_LCP: k[e] = lcp_priority(ctx, L, e); break;
      case MS_CACHE_LRU: k[e] = static_cast<double>(L.last_use[e]); break;
      case MS_CACHE_LFU: k[e] = L.mu[e]; break;
      default: k[e] = static_cast<double>(next_random(ctx) >> 11); break;
    }
  }
  return k;
}

void set_route_workspace(ms_ctx* ctx, msk::RouteArgs* r) {
  const Shape& s = ctx->s;
  r->lrank = reinterpret_cast<int32_t*>(ctx->dev(s.off_lrank));
  r->blk = reinterpret_cast<int32_t*>(ctx->dev(s.off_blk));
  r->psc = reinterpret_cast<float*>(ctx->dev(s.off_psc));
  r->nblk_cap = s.nblk_cap;
}

// Order work on `stream` after the previous forward/prediction of this
// context (they share the work buffers).
ms_status flush_fwd(ms_ctx* ctx, LayerState& L);
ms_status flush_all_fwd(ms_ctx* ctx);
ms_status order_after_last(ms_ctx* ctx, hipStream_t stream) {
  if (ctx->has_last && ctx->last_stream != stream) {
    const ms_status st = flush_all_fwd(ctx);
    if (st != MS_OK) return st;
    MS_HIP(hipStreamWaitEvent(stream, ctx->last_ev, 0));
  }
  return MS_OK;
}

// Record a layer's end-of-forward event left unrecorded (recorded now, it
// marks at least the end of that forward), and every layer's.
ms_status flush_fwd(ms_ctx* ctx, LayerState& L) {
  if (L.fwd_unrecorded) {
    MS_HIP(hipEventRecord(L.last_fwd, L.fwd_stream));
    L.fwd_unrecorded = false;
  }
  return MS_OK;
}
ms_status flush_all_fwd(ms_ctx* ctx) {
  for (LayerState& L : ctx->layers) {
    const ms_status st = flush_fwd(ctx, L);
    if (st != MS_OK) return st;
  }
  return MS_OK;
}

// Prefill path of one forward, after the host has the routing (offsets).
// Matrix-core gate/up writes bf16 activations per routed slot (and per token
// for shared experts); the down projection runs once all of an expert's
// chunks are in VRAM and writes the slot's single partial plane.
//   compute stream: gate/up over cached tops, staging groups that already
//     landed and shared experts; then the down projection of every expert
//     now complete in VRAM and of the shared experts;
//   side stream (after that gate/up): per expert with missing chunks, issue
//     the copies, gate/up per group as it lands, then its down projection,
//     then release its staging slot.
// gate + up and down bytes of one chunk (b-bit: codes and their metadata)
uint64_t mma_gu_bytes(const Shape& s) {
  return s.bits ? 2 * (msk::q_off_uq(s.d, s.bits) + 4ull * s.d) : 2ull * kUnits * s.d * s.elem;
}
uint64_t mma_dn_bytes(const Shape& s) {
  return s.bits ? msk::q_off_uq(s.d, s.bits) + 4ull * s.d : 1ull * kUnits * s.d * s.elem;
}

// The fields of the matrix-core kernels' arguments that every launch of a
// forward shares.
void mma_common(ms_ctx* ctx, const void* h_dev, int T, msk::MmaArgs& ma) {
  const Shape& s = ctx->s;
  ma.h = h_dev;
  ma.offsets = reinterpret_cast<const int32_t*>(ctx->dev(s.off_offsets));
  ma.perm = reinterpret_cast<const int32_t*>(ctx->dev(s.off_perm));
  ma.act = reinterpret_cast<uint16_t*>(ctx->dev(s.off_act));
  ma.act_sh = reinterpret_cast<uint16_t*>(ctx->dev(s.off_act_sh));
  ma.part = reinterpret_cast<float*>(ctx->dev(s.off_part));
  ma.part_sh = reinterpret_cast<float*>(ctx->dev(s.off_part_sh));
  ma.chunk_bytes = s.chunk_bytes;
  ma.sh_plane = s.sh_plane;
  ma.d = s.d;
  ma.K = s.K;
  ma.T = T;
  ma.f_pad = s.n_chunks * kUnits;
  ma.f_pad_sh = s.n_chunks_sh * kUnits;
  ma.rows_shared = s.max_T;
  ma.ncb = (s.d + msk::kMmaCols - 1) / msk::kMmaCols;
  ma.bits = s.bits;
  ma.ksplit = s.down_splits;
}

// Whether the resident part of a prefill forward is planned on the device
// (LDS-staged kernels for both projections, a task per expert within the
// plan kernel's reach).
bool plan_on_device(const Shape& s) {
  return s.bits == 0 && s.dtype == MS_BF16 && s.d % msk::kMmaCols == 0 && s.n_sh <= msk::kMaxPlanShared &&
         s.E + s.n_sh <= msk::kMaxPlanTasks;
}

// Launch the plan, then the resident experts' gate/up and down over it, on
// sm right after the routing (work-groups past the planned ones exit).
// Returns the timeline records of the two launches (bytes set once the
// routing is known).
ms_status launch_planned(ms_ctx* ctx, int layer, const void* h_dev, int T, hipStream_t sm, int* tl_gu, int* tl_dn) {
  const Shape& s = ctx->s;
  LayerState& L = ctx->layers[layer];
  msk::PlanArgs pa{};
  auto* plan = reinterpret_cast<msk::MmaTask*>(ctx->dev(s.off_plan));
  auto* counts = reinterpret_cast<int32_t*>(plan + 2 * msk::kMaxPlanTasks);
  pa.offsets = reinterpret_cast<const int32_t*>(ctx->dev(s.off_offsets));
  pa.gu = plan;
  pa.dn = plan + msk::kMaxPlanTasks;
  pa.counts = counts;
  pa.cache_base = L.cache_base;
  pa.top_bytes = L.top_bytes;
  for (int i = 0; i < s.n_sh; ++i)
    pa.shared[i] = ctx->dev(s.off_shared + align_up(s.shared_bytes, kAlign) * (static_cast<uint64_t>(layer) * s.n_sh + i));
  pa.E = s.E;
  pa.T = T;
  pa.n_chunks = s.n_chunks;
  pa.n_chunks_sh = s.n_chunks_sh;
  pa.n_sh = s.n_sh;
  pa.ncb = (s.d + msk::kMmaCols - 1) / msk::kMmaCols;
  pa.tile_rows = msk::kGdMaxRows;
  // upper bounds of the work-groups: sum over experts of resident chunks x
  // ceil(rows / tile) <= resident chunks + chunks x ceil(T K / tile)
  const int extra_tiles = static_cast<int>((static_cast<int64_t>(T) * s.K + msk::kGdMaxRows - 1) / msk::kGdMaxRows);
  const int sh_tiles = (T + msk::kGdMaxRows - 1) / msk::kGdMaxRows;
  int64_t gu_wg = static_cast<int64_t>(s.n_chunks) * extra_tiles + static_cast<int64_t>(s.n_sh) * sh_tiles * s.n_chunks_sh;
  int64_t n_full = 0;
  for (int e = 0; e < s.E; ++e) {
    const int rc = resident_chunks(L, e);
    pa.res[e] = static_cast<int16_t>(rc);
    pa.slot[e] = static_cast<int16_t>(rc > 0 ? L.slot_of[e] : 0);
    gu_wg += rc;
    n_full += rc >= s.n_chunks;
  }
  const int64_t dn_wg = (n_full + extra_tiles + static_cast<int64_t>(s.n_sh) * sh_tiles) * pa.ncb;
  MS_HIP(msk::launch_prefill_plan(pa, sm));
  msk::MmaArgs ma{};
  mma_common(ctx, h_dev, T, ma);
  ma.tile_rows = msk::kGdMaxRows;
  ma.gu_split = 1;
  ma.dtasks = pa.gu;
  ma.dcount = counts;
  ma.n_wg = static_cast<int>(std::min<int64_t>(gu_wg, INT32_MAX));
  *tl_gu = tl_begin(ctx, sm, MS_IV_FFN_RESIDENT, layer, 0);
  MS_HIP(msk::launch_mma_gateup(ma, sm));
  tl_end(ctx, *tl_gu, sm);
  ma.dtasks = pa.dn;
  ma.dcount = counts + 2;
  ma.n_wg = static_cast<int>(std::min<int64_t>(dn_wg, INT32_MAX));
  *tl_dn = tl_begin(ctx, sm, MS_IV_FFN_DOWN, layer, 0);
  MS_HIP(msk::launch_mma_down(ma, sm));
  tl_end(ctx, *tl_dn, sm);
  return MS_OK;
}

// Prefill experts once the routing is known.  With `planned`, the resident
// chunks' gate/up, the down of fully resident experts and the shared experts
// were launched before (launch_planned); the rest goes here.
ms_status prefill_experts(ms_ctx* ctx, int layer, const void* h_dev, int T, const std::vector<int32_t>& offs,
                          hipStream_t sm, bool planned) {
  const Shape& s = ctx->s;
  LayerState& L = ctx->layers[layer];
  const uint64_t gu_bytes = mma_gu_bytes(s);
  const uint64_t dn_bytes = mma_dn_bytes(s);
  msk::MmaArgs ma{};
  mma_common(ctx, h_dev, T, ma);
  auto m_tiles = [&](int e) {
    const int n = e >= 0 ? offs[e + 1] - offs[e] : T;
    return (n + msk::kMmaRows - 1) / msk::kMmaRows;
  };
  auto shared_base = [&](int i) {
    return ctx->dev(s.off_shared + align_up(s.shared_bytes, kAlign) * (static_cast<uint64_t>(layer) * s.n_sh + i));
  };
  auto rows_of = [&](int e) { return e >= 0 ? offs[e + 1] - offs[e] : T; };
  auto launch_group = [&](const std::vector<msk::MmaTask>& tasks, hipStream_t st, bool down,
                          int tile_rows) -> ms_status {
    ma.tile_rows = tile_rows;
    for (size_t i0 = 0; i0 < tasks.size(); i0 += msk::kMaxMmaTasks) {
      const size_t i1 = std::min(tasks.size(), i0 + msk::kMaxMmaTasks);
      ma.n_tasks = static_cast<int>(i1 - i0);
      int tiles = 0;
      for (size_t i = i0; i < i1; ++i) tiles += tasks[i].m_tiles * tasks[i].n_chunks;
      ma.gu_split = (tile_rows == msk::kMmaRows && tiles < msk::kGuSplitBelow && s.bits == 0) ? 4 : 1;
      int wg = 0;
      uint64_t bytes = 0;
      for (size_t i = i0; i < i1; ++i) {
        ma.tasks[i - i0] = tasks[i];
        ma.tasks[i - i0].wg_begin = wg;
        // (the LDS-staged gate/up kernel takes gd_group_chunks chunks per work-group)
        const bool staged = !down && s.bits == 0 && ma.gu_split == 1 && s.d % 128 == 0;
        const int gc = msk::gd_group_chunks(rows_of(tasks[i].expert), tasks[i].n_chunks);
        const int per = staged ? (tasks[i].n_chunks + gc - 1) / gc : tasks[i].n_chunks * ma.gu_split;
        wg += tasks[i].m_tiles * (down ? ma.ncb * ma.ksplit : per);
        bytes += (down ? dn_bytes : gu_bytes) * tasks[i].n_chunks;
      }
      ma.n_wg = wg;
      const int id = tl_begin(ctx, st, down ? MS_IV_FFN_DOWN : (st == sm ? MS_IV_FFN_RESIDENT : MS_IV_FFN_STREAMED),
                              layer, bytes);
      MS_HIP(down ? msk::launch_mma_down(ma, st) : msk::launch_mma_gateup(ma, st));
      tl_end(ctx, id, st);
    }
    return MS_OK;
  };
  // bf16 gate/up with d % 128 == 0: row tiles of up to kGdMaxRows rows, so
  // that an expert's rows usually fit one tile and its weights are read once
  // (the kernel sizes each work-group to its tile), when those tiles fill the
  // GPU; otherwise 64-row tiles, split four ways per chunk when even those
  // are few.  The tile height changes no result.
  // The bf16 down projection with d % kMmaCols == 0 always takes such tiles.
  auto launch = [&](const std::vector<msk::MmaTask>& tasks, hipStream_t st, bool down) -> ms_status {
    if (s.bits != 0 || s.d % (down ? msk::kMmaCols : 128) != 0) return launch_group(tasks, st, down, msk::kMmaRows);
    std::vector<msk::MmaTask> tall = tasks;
    int tiles = 0;
    for (msk::MmaTask& t : tall) {
      t.m_tiles = (rows_of(t.expert) + msk::kGdMaxRows - 1) / msk::kGdMaxRows;
      tiles += t.m_tiles * t.n_chunks;
    }
    if (!down && tiles < msk::kGuSplitBelow) return launch_group(tasks, st, false, msk::kMmaRows);
    return launch_group(tall, st, down, msk::kGdMaxRows);
  };
  auto task = [](const unsigned char* base, const unsigned char* base2, int e, int lo, int n, int split, int mt) {
    msk::MmaTask t{};
    t.base = base;
    t.base2 = base2;
    t.expert = e;
    t.chunk_lo = lo;
    t.n_chunks = n;
    t.split = split;
    t.m_tiles = mt;
    return t;
  };

  // statistics and, per active expert, whether all its chunks are in VRAM now
  std::vector<int> covering(s.E, -1);
  std::vector<char> complete(s.E, 0);
  int use_counter = 0;
  std::vector<msk::MmaTask> gu, dn;
  for (int e = 0; e < s.E; ++e) {
    if (offs[e + 1] == offs[e]) continue;
    L.st.experts_active += 1;
    const int res = resident_chunks(L, e);
    const unsigned char* top = res > 0 ? L.cache_base + L.top_bytes * L.slot_of[e] : nullptr;
    if (res > 0 && !planned) gu.push_back(task(top, nullptr, e, 0, res, 0, m_tiles(e)));
    if (res >= s.n_chunks) {
      L.st.alpha += 1;
      complete[e] = 1;
      if (!planned) dn.push_back(task(top, top, e, 0, s.n_chunks, s.n_chunks, m_tiles(e)));
      continue;
    }
    if (res > 0)
      L.st.beta += 1;
    else
      L.st.gamma += 1;
    const int si = find_slot(ctx, layer, e);
    if (si < 0 || ctx->buf[si].first_chunk > res) continue;
    covering[e] = si;
    BufSlot& b = ctx->buf[si];
    bool any_issued = false, all_landed = true;
    for (int gi = 0; gi < static_cast<int>(b.groups.size()); ++gi) {
      Group& g = b.groups[gi];
      any_issued = any_issued || g.issued;
      const int lo = std::max(g.c_lo, res);
      if (lo >= g.c_hi) continue;
      const hipError_t q = group_landed(ctx, si, gi);
      if (q != hipSuccess && q != hipErrorNotReady) return poison(ctx, "hipEventQuery(group)", q);
      if (q == hipSuccess) {
        gu.push_back(task(b.base, nullptr, e, lo, g.c_hi - lo, 0, m_tiles(e)));
        g.pre = true;
        if (g.prefetch && !g.used) L.st.bytes_prefetch_used += s.chunk_bytes * (g.c_hi - g.c_lo);
        g.used = true;
      } else {
        all_landed = false;
      }
    }
    if (any_issued) L.st.buffer_hits += 1;
    if (all_landed) {
      complete[e] = 1;
      dn.push_back(task(top ? top : b.base, b.base, e, 0, s.n_chunks, res, m_tiles(e)));
      b.use_order = use_counter++;  // read first, by the compute stream
    }
  }
  for (int i = 0; i < s.n_sh && !planned; ++i) {
    gu.push_back(task(shared_base(i), nullptr, -1 - i, 0, s.n_chunks_sh, 0, m_tiles(-1)));
    dn.push_back(task(shared_base(i), shared_base(i), -1 - i, 0, s.n_chunks_sh, s.n_chunks_sh, m_tiles(-1)));
  }
  // the side streams below need the resident gate/up only if an expert is
  // still missing chunks (a marker between kernels costs the stream a few
  // microseconds)
  bool any_missing = false;
  for (int e = 0; e < s.E && !any_missing; ++e) any_missing = offs[e + 1] > offs[e] && !complete[e];
  ms_status st = launch(gu, sm, false);
  if (st != MS_OK) return st;
  if (any_missing) MS_HIP(hipEventRecord(ctx->ev_res, sm));
  st = launch(dn, sm, true);
  if (st != MS_OK) return st;
  for (int e = 0; e < s.E; ++e) {
    if (covering[e] >= 0 && complete[e]) {
      BufSlot& b = ctx->buf[covering[e]];
      MS_HIP(hipEventRecord(b.last_read, sm));
      b.has_last_read = true;
    }
  }

  // experts still missing chunks: side stream, those a staging slot already
  // covers first.  Their slots stay reserved until then, so that no other
  // miss evicts them.
  // Missing experts alternate between two side streams: each expert's
  // launches are small (a few row tiles), so two run side by side.
  if (!any_missing) return MS_OK;
  MS_HIP(hipStreamWaitEvent(ctx->side, ctx->ev_res, 0));
  MS_HIP(hipStreamWaitEvent(ctx->side2, ctx->ev_res, 0));
  for (int e = 0; e < s.E; ++e)
    if (covering[e] >= 0 && !complete[e]) ctx->buf[covering[e]].use_order = kReserved;
  int n_missing = 0;
  for (const int e : miss_order(ctx, layer, offs, &complete)) {
    hipStream_t ss = (n_missing++ % 2) ? ctx->side2 : ctx->side;
    const int res = resident_chunks(L, e);
    int si = covering[e];
    if (si < 0) {
      // a slot of (layer, e) that starts above the resident part (its top
      // was evicted since) is reassigned, as on the decode path, so that no
      // two slots ever hold the same expert
      si = find_slot(ctx, layer, e);
      if (si < 0) si = pick_victim(ctx, true);
      if (si < 0) return fail(ctx, MS_E_STATE, "no staging slot can be taken");
      st = assign_slot(ctx, si, layer, e, res, true);
      if (st != MS_OK) return st;
    }
    BufSlot& b = ctx->buf[si];
    b.use_order = use_counter++;
    b.tick = ++ctx->tick;
    for (int gi = 0; gi < static_cast<int>(b.groups.size()); ++gi) {
      Group& g = b.groups[gi];
      const int lo = std::max(g.c_lo, res);
      if (lo >= g.c_hi || g.pre) continue;
      if (!g.issued) {
        st = issue_group(ctx, si, gi, false);
        if (st != MS_OK) return st;
      } else if (g.prefetch && !g.used) {
        L.st.bytes_prefetch_used += s.chunk_bytes * (g.c_hi - g.c_lo);
      }
      g.used = true;
      MS_HIP(hipStreamWaitEvent(ss, b.gev[gi], 0));
      (ss == ctx->side ? ctx->side_work : ctx->side2_work) = true;
      st = launch({task(b.base, nullptr, e, lo, g.c_hi - lo, 0, m_tiles(e))}, ss, false);
      if (st != MS_OK) return st;
    }
    const unsigned char* top = res > 0 ? L.cache_base + L.top_bytes * L.slot_of[e] : b.base;
    (ss == ctx->side ? ctx->side_work : ctx->side2_work) = true;
    st = launch({task(top, b.base, e, 0, s.n_chunks, res, m_tiles(e))}, ss, true);
    if (st != MS_OK) return st;
    MS_HIP(hipEventRecord(b.last_read, ss));
    b.has_last_read = true;
  }
  return MS_OK;
}

}  // namespace

// ============================================================== C ABI ====

extern "C" {

ms_status ms_query_sizes(const ms_model_desc* desc, ms_sizes* out) {
  if (!out) return MS_E_INVALID;
  Shape s;
  std::string err;
  ms_status st = derive_shape(desc, &s, &err);
  if (st != MS_OK) return st;
  out->chunk_bytes = s.chunk_bytes;
  out->n_chunks = s.n_chunks;
  out->expert_bytes = s.expert_bytes;
  out->fixed_pool_bytes = s.fixed_bytes;
  out->buffer_bytes = s.expert_bytes * s.n_buf;
  return MS_OK;
}

ms_status ms_split_plan(const ms_model_desc* desc, uint64_t budget_bytes, float r, int32_t* top_units_out,
                        uint64_t* top_bytes_out, int32_t* top_slots_out) {
  Shape s;
  std::string err;
  ms_status st = derive_shape(desc, &s, &err);
  if (st != MS_OK) return st;
  if (!(r >= 0.0f && r <= 1.0f)) return MS_E_INVALID;
  const int units = top_units_for(r, s.F);
  const int chunks = (units + kUnits - 1) / kUnits;
  const uint64_t tb = s.chunk_bytes * chunks;
  int32_t slots = 0;
  if (tb > 0) slots = static_cast<int32_t>(std::min<uint64_t>(budget_bytes / tb, s.E));
  if (top_units_out) *top_units_out = units;
  if (top_bytes_out) *top_bytes_out = tb;
  if (top_slots_out) *top_slots_out = slots;
  return MS_OK;
}

const char* ms_last_error(const ms_ctx* ctx) { return ctx ? ctx->err.c_str() : "NULL context"; }

ms_status ms_create(const ms_model_desc* desc, void* dev_pool, uint64_t pool_bytes, int32_t host_store_experts,
                    ms_ctx** out) {
  if (!out) return MS_E_INVALID;
  *out = nullptr;
  ms_ctx* ctx = new ms_ctx();
  std::string err;
  ms_status st = derive_shape(desc, &ctx->s, &err);
  if (st != MS_OK) {
    delete ctx;
    return st;
  }
  if (!dev_pool || (reinterpret_cast<uintptr_t>(dev_pool) % kAlign) != 0) {
    delete ctx;
    return MS_E_INVALID;
  }
  if (pool_bytes < ctx->s.fixed_bytes) {
    delete ctx;
    return MS_E_BUDGET;
  }
  if (host_store_experts < 0) {
    delete ctx;
    return MS_E_INVALID;
  }
  ctx->pool = static_cast<unsigned char*>(dev_pool);
  ctx->pool_bytes = pool_bytes;
  ctx->blob_cap = host_store_experts;
  const Shape& s = ctx->s;
  auto cleanup_fail = [&](hipError_t e, const char* what) {
    ms_status rs = poison(ctx, what, e);
    (void)rs;
    ms_destroy(ctx);
    return MS_E_HIP;
  };
  hipError_t e;
  if ((e = hipGetDevice(&ctx->device)) != hipSuccess) return cleanup_fail(e, "hipGetDevice");
  if ((e = scratch_address(ctx->device, &ctx->scratch_addr)) != hipSuccess)
    return cleanup_fail(e, "hipGetSymbolAddress(scratch)");
  if ((e = hipStreamCreateWithFlags(&ctx->copy, hipStreamNonBlocking)) != hipSuccess)
    return cleanup_fail(e, "hipStreamCreate(copy)");
  if ((e = hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking)) != hipSuccess)
    return cleanup_fail(e, "hipStreamCreate(side)");
  if ((e = hipStreamCreateWithFlags(&ctx->side2, hipStreamNonBlocking)) != hipSuccess)
    return cleanup_fail(e, "hipStreamCreate(side2)");
  for (hipEvent_t* ev : {&ctx->ev_route, &ctx->ev_res, &ctx->ev_side_done, &ctx->ev_last, &ctx->ev_side2_done})
    if ((e = hipEventCreateWithFlags(ev, hipEventDisableTiming)) != hipSuccess)
      return cleanup_fail(e, "hipEventCreate");
  // small host buffers that kernels write directly (mapped, coherent)
  const unsigned mflags = hipHostMallocMapped | hipHostMallocCoherent;
  if ((e = hipHostMalloc(reinterpret_cast<void**>(&ctx->h_offsets), sizeof(int32_t) * (s.E + 1), mflags)) != hipSuccess)
    return cleanup_fail(e, "hipHostMalloc(offsets)");
  if ((e = hipHostMalloc(reinterpret_cast<void**>(&ctx->h_order), sizeof(int32_t) * s.E, mflags)) != hipSuccess)
    return cleanup_fail(e, "hipHostMalloc(order)");
  if ((e = hipHostMalloc(reinterpret_cast<void**>(&ctx->h_score), sizeof(float) * s.E, mflags)) != hipSuccess)
    return cleanup_fail(e, "hipHostMalloc(score)");
  if ((e = hipHostGetDevicePointer(reinterpret_cast<void**>(&ctx->d_offsets_map), ctx->h_offsets, 0)) != hipSuccess)
    return cleanup_fail(e, "hipHostGetDevicePointer(offsets)");
  if ((e = hipHostGetDevicePointer(reinterpret_cast<void**>(&ctx->d_order_map), ctx->h_order, 0)) != hipSuccess)
    return cleanup_fail(e, "hipHostGetDevicePointer(order)");
  if ((e = hipHostGetDevicePointer(reinterpret_cast<void**>(&ctx->d_score_map), ctx->h_score, 0)) != hipSuccess)
    return cleanup_fail(e, "hipHostGetDevicePointer(score)");
  if ((e = hipHostMalloc(reinterpret_cast<void**>(&ctx->h_seq), sizeof(int32_t), mflags)) != hipSuccess)
    return cleanup_fail(e, "hipHostMalloc(seq)");
  *reinterpret_cast<volatile int32_t*>(ctx->h_seq) = 0;
  if ((e = hipHostGetDevicePointer(reinterpret_cast<void**>(&ctx->d_seq_map), ctx->h_seq, 0)) != hipSuccess)
    return cleanup_fail(e, "hipHostGetDevicePointer(seq)");
  ctx->layers.resize(s.L);
  for (LayerState& L : ctx->layers) {
    L.blob_of.assign(s.E, -1);
    L.shared_set.assign(s.n_sh, false);
    L.slot_of.assign(s.E, -1);
    L.mu.assign(s.E, 0.0);
    L.nu.assign(s.E, 0.0);
    L.last_use.assign(s.E, 0);
    L.hit_hist.assign(s.E, 0);
    L.pred_act.assign(s.E, 0);
    L.pred_rank.assign(static_cast<size_t>(s.E) * s.E, 0);
    if ((e = hipEventCreateWithFlags(&L.last_fwd, hipEventDisableTiming)) != hipSuccess)
      return cleanup_fail(e, "hipEventCreate(layer)");
  }
  ctx->buf.resize(s.n_buf);
  // one completion event per copy group a slot can hold: a slot's content is
  // cut into at most ceil(n_chunks / group size) groups (assign_slot), so
  // no forward ever creates one
  const int g_min = std::max(1, std::min(s.group_chunks, s.miss_group_chunks));
  const int max_groups = (s.n_chunks + g_min - 1) / g_min;
  for (int i = 0; i < s.n_buf; ++i) {
    ctx->buf[i].base = ctx->dev(s.off_buffer + s.expert_bytes * i);
    if ((e = hipEventCreateWithFlags(&ctx->buf[i].last_read, hipEventDisableTiming)) != hipSuccess)
      return cleanup_fail(e, "hipEventCreate(slot)");
    for (int g = 0; g < max_groups; ++g) {
      hipEvent_t ev;
      if ((e = hipEventCreateWithFlags(&ev, hipEventDisableTiming)) != hipSuccess)
        return cleanup_fail(e, "hipEventCreate(copy group)");
      ctx->buf[i].gev.push_back(ev);
    }
  }
  *out = ctx;
  return MS_OK;
}

void ms_destroy(ms_ctx* ctx) {
  if (!ctx) return;
  if (ctx->copy) (void)hipStreamSynchronize(ctx->copy);
  if (ctx->side) (void)hipStreamSynchronize(ctx->side);
  if (ctx->side2) (void)hipStreamSynchronize(ctx->side2);
  (void)flush_all_fwd(ctx);
  if (ctx->has_last) (void)hipEventSynchronize(ctx->last_ev);
  for (LayerState& L : ctx->layers) {
    for (hipEvent_t ev : L.pending_loads) (void)hipEventDestroy(ev);
    if (L.last_fwd) (void)hipEventDestroy(L.last_fwd);
  }
  for (BufSlot& b : ctx->buf) {
    for (hipEvent_t ev : b.gev) (void)hipEventDestroy(ev);
    if (b.last_read) (void)hipEventDestroy(b.last_read);
  }
  for (hipEvent_t ev : ctx->free_events) (void)hipEventDestroy(ev);
  for (TlRec& r : ctx->tl) {
    (void)hipEventDestroy(r.e0);
    (void)hipEventDestroy(r.e1);
  }
  for (hipEvent_t ev : ctx->tl_pool) (void)hipEventDestroy(ev);
  if (ctx->tl_origin) (void)hipEventDestroy(ctx->tl_origin);
  for (hipEvent_t ev : {ctx->ev_route, ctx->ev_res, ctx->ev_side_done, ctx->ev_last, ctx->ev_side2_done})
    if (ev) (void)hipEventDestroy(ev);
  for (unsigned char* p : ctx->blobs) (void)hipHostFree(p);
  if (ctx->h_offsets) (void)hipHostFree(ctx->h_offsets);
  if (ctx->h_order) (void)hipHostFree(ctx->h_order);
  if (ctx->h_score) (void)hipHostFree(ctx->h_score);
  if (ctx->h_seq) (void)hipHostFree(ctx->h_seq);
  if (ctx->copy) (void)hipStreamDestroy(ctx->copy);
  if (ctx->side) (void)hipStreamDestroy(ctx->side);
  if (ctx->side2) (void)hipStreamDestroy(ctx->side2);
  delete ctx;
}

ms_status ms_set_router(ms_ctx* ctx, int32_t layer, const void* w_r, const float* bias) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  if (!w_r) return fail(ctx, MS_E_INVALID, "w_r is NULL");
  const Shape& s = ctx->s;
  MS_HIP(hipMemcpy(ctx->dev(s.off_router + s.router_stride * layer), w_r,
                   static_cast<size_t>(s.d) * s.E * s.elem, hipMemcpyHostToDevice));
  {
    // transposed copy [E][d] for the many-token logits kernel
    std::vector<unsigned char> wt(static_cast<size_t>(s.d) * s.E * s.elem);
    const unsigned char* src = static_cast<const unsigned char*>(w_r);
    for (int j = 0; j < s.d; ++j)
      for (int e = 0; e < s.E; ++e)
        std::memcpy(&wt[(static_cast<size_t>(e) * s.d + j) * s.elem], src + (static_cast<size_t>(j) * s.E + e) * s.elem,
                    s.elem);
    MS_HIP(hipMemcpy(ctx->dev(s.off_router_t + s.router_stride * layer), wt.data(), wt.size(), hipMemcpyHostToDevice));
  }
  LayerState& L = ctx->layers[layer];
  if (bias) MS_HIP(hipMemcpy(ctx->dev(s.off_bias + s.bias_stride * layer), bias, sizeof(float) * s.E,
                             hipMemcpyHostToDevice));
  L.router_set = true;
  L.bias_set = bias != nullptr;
  return MS_OK;
}

// Write expert (layer, e)'s host blob with `pack` (called with the blob),
// allocating it unless the expert owns one alone; then drop staged copies of
// the old contents and copy cached top segments again.
static ms_status write_expert_blob(ms_ctx* ctx, int32_t layer, int32_t e,
                                   const std::function<void(unsigned char*)>& pack) {
  ms_status st = MS_OK;
  const Shape& s = ctx->s;
  LayerState& L = ctx->layers[layer];
  int bi = L.blob_of[e];
  // reuse the blob only if no other (layer, expert) aliases it
  if (bi >= 0) {
    int users = 0;
    for (const LayerState& L2 : ctx->layers)
      for (int b : L2.blob_of) users += (b == bi);
    if (users > 1) bi = -1;
  }
  if (bi < 0) {
    if (ctx->blob_cap > 0 && static_cast<int>(ctx->blobs.size()) >= ctx->blob_cap)
      return fail(ctx, MS_E_NOMEM, "host expert store is full (host_store_experts)");
    // coherent: the copy kernel reads it over PCIe uncached, so a blob
    // rewritten (or freed and reallocated) later is never read stale
    void* p = nullptr;
    hipError_t he = hipHostMalloc(&p, s.expert_bytes, hipHostMallocCoherent);
    if (he != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(ctx, MS_E_NOMEM, "hipHostMalloc of an expert blob failed");
    }
    void* pd = nullptr;
    he = hipHostGetDevicePointer(&pd, p, 0);
    if (he != hipSuccess || !pd) {
      (void)hipGetLastError();
      (void)hipHostFree(p);
      return fail(ctx, MS_E_NOMEM, "expert blob has no device address");
    }
    ctx->blobs.push_back(static_cast<unsigned char*>(p));
    ctx->blobs_dev.push_back(static_cast<unsigned char*>(pd));
    bi = static_cast<int>(ctx->blobs.size()) - 1;
  }
  // the blob may be read by work in flight: drain it before rewriting
  st = ms_sync(ctx);
  if (st != MS_OK) return st;
  pack(ctx->blobs[bi]);
  L.blob_of[e] = bi;
  // copies of the old weights: staging slots are dropped (with any queued
  // prefetch), cached top segments are copied again
  ctx->pf_queue.clear();
  ctx->pf_inflight.clear();
  for (BufSlot& b : ctx->buf)
    if (b.layer >= 0 && ctx->layers[b.layer].blob_of[b.expert] == bi) clear_slot(b);
  for (int l = 0; l < s.L; ++l) {
    LayerState& L2 = ctx->layers[l];
    for (int e2 = 0; e2 < s.E; ++e2) {
      if (L2.blob_of[e2] != bi || L2.slot_of[e2] < 0) continue;
      st = issue_copy(ctx, L2.cache_base + L2.top_bytes * L2.slot_of[e2], ctx->blobs[bi], ctx->blobs_dev[bi],
                      L2.top_bytes, MS_IV_COPY_TOP, l);
      if (st != MS_OK) return st;
      hipEvent_t ev;
      MS_HIP(new_event(ctx, &ev));
      MS_HIP(hipEventRecord(ev, ctx->copy));
      L2.pending_loads.push_back(ev);
    }
  }
  return MS_OK;
}

ms_status ms_set_expert(ms_ctx* ctx, int32_t layer, int32_t e, const void* w_gate, const void* w_up,
                        const void* w_down) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  const Shape& s = ctx->s;
  if (e < 0 || e >= s.E) return fail(ctx, MS_E_INVALID, "expert out of range");
  if (!w_gate || !w_up || !w_down) return fail(ctx, MS_E_INVALID, "weight pointer is NULL");
  if (s.bits != 0) return fail(ctx, MS_E_STATE, "this model's experts are b-bit codes (ms_set_expert_q)");
  return write_expert_blob(ctx, layer, e, [&](unsigned char* blob) {
    pack_expert(w_gate, w_up, w_down, s.d, s.F, s.n_chunks, s.elem, blob);
  });
}

ms_status ms_set_expert_q(ms_ctx* ctx, int32_t layer, int32_t e, const void* gate_q, const void* gate_m,
                          const void* up_q, const void* up_m, const void* down_q, const void* down_m) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  const Shape& s = ctx->s;
  if (e < 0 || e >= s.E) return fail(ctx, MS_E_INVALID, "expert out of range");
  if (!gate_q || !gate_m || !up_q || !up_m || !down_q || !down_m)
    return fail(ctx, MS_E_INVALID, "code or metadata pointer is NULL");
  if (s.bits == 0) return fail(ctx, MS_E_STATE, "this model's experts are not b-bit codes (ms_set_expert)");
  return write_expert_blob(ctx, layer, e, [&](unsigned char* blob) {
    pack_expert_q(static_cast<const uint8_t*>(gate_q), static_cast<const uint16_t*>(gate_m),
                  static_cast<const uint8_t*>(up_q), static_cast<const uint16_t*>(up_m),
                  static_cast<const uint8_t*>(down_q), static_cast<const uint16_t*>(down_m), s.d, s.F, s.bits, blob);
  });
}

ms_status ms_alias_expert(ms_ctx* ctx, int32_t layer, int32_t e, int32_t src_layer, int32_t src_e) {
  MS_CHECK_CTX(ctx);
  if (check_layer(ctx, layer) != MS_OK || check_layer(ctx, src_layer) != MS_OK)
    return fail(ctx, MS_E_INVALID, "layer out of range");
  const Shape& s = ctx->s;
  if (e < 0 || e >= s.E || src_e < 0 || src_e >= s.E) return fail(ctx, MS_E_INVALID, "expert out of range");
  const int bi = ctx->layers[src_layer].blob_of[src_e];
  if (bi < 0) return fail(ctx, MS_E_STATE, "source expert not set");
  ctx->layers[layer].blob_of[e] = bi;
  return MS_OK;
}

ms_status ms_set_shared_expert(ms_ctx* ctx, int32_t layer, int32_t sidx, const void* w_gate, const void* w_up,
                               const void* w_down) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  const Shape& s = ctx->s;
  if (sidx < 0 || sidx >= s.n_sh) return fail(ctx, MS_E_INVALID, "shared expert out of range");
  if (!w_gate || !w_up || !w_down) return fail(ctx, MS_E_INVALID, "weight pointer is NULL");
  std::vector<unsigned char> tmp(s.shared_bytes);
  pack_expert(w_gate, w_up, w_down, s.d, s.F_sh, s.n_chunks_sh, s.elem, tmp.data());
  const uint64_t off = s.off_shared + align_up(s.shared_bytes, kAlign) * (static_cast<uint64_t>(layer) * s.n_sh + sidx);
  st = flush_all_fwd(ctx);
  if (st != MS_OK) return st;
  if (ctx->has_last) MS_HIP(hipEventSynchronize(ctx->last_ev));
  MS_HIP(hipMemcpy(ctx->dev(off), tmp.data(), s.shared_bytes, hipMemcpyHostToDevice));
  ctx->layers[layer].shared_set[sidx] = true;
  return MS_OK;
}

ms_status ms_sync(ms_ctx* ctx) {
  MS_CHECK_CTX(ctx);
  MS_HIP(hipStreamSynchronize(ctx->copy));
  MS_HIP(hipStreamSynchronize(ctx->side));
  MS_HIP(hipStreamSynchronize(ctx->side2));
  const ms_status st = flush_all_fwd(ctx);
  if (st != MS_OK) return st;
  if (ctx->has_last) MS_HIP(hipEventSynchronize(ctx->last_ev));
  return MS_OK;
}

ms_status ms_configure(ms_ctx* ctx, const uint64_t* budget_bytes, const float* r, int32_t* top_slots_out) {
  MS_CHECK_CTX(ctx);
  if (!budget_bytes || !r) return fail(ctx, MS_E_INVALID, "NULL budget or ratio array");
  const Shape& s = ctx->s;
  uint64_t total = 0;
  for (int i = 0; i < s.L; ++i) {
    if (!(r[i] >= 0.0f && r[i] <= 1.0f)) return fail(ctx, MS_E_INVALID, "split ratio outside [0, 1]");
    total += budget_bytes[i];
  }
  if (total > ctx->pool_bytes - s.fixed_bytes)
    return fail(ctx, MS_E_BUDGET, "sum of layer budgets exceeds the device pool");
  ms_status st = ms_sync(ctx);
  if (st != MS_OK) return st;
  ctx->pf_queue.clear();
  ctx->pf_inflight.clear();
  for (BufSlot& b : ctx->buf) {
    clear_slot(b);
    b.has_last_read = false;
    b.use_order = -1;
  }
  uint64_t off = s.fixed_bytes;
  for (int i = 0; i < s.L; ++i) {
    LayerState& L = ctx->layers[i];
    L.budget = budget_bytes[i];
    L.r = r[i];
    L.top_units = top_units_for(r[i], s.F);
    L.top_chunks = (L.top_units + kUnits - 1) / kUnits;
    L.top_bytes = s.chunk_bytes * L.top_chunks;
    L.slots = L.top_bytes > 0 ? static_cast<int>(std::min<uint64_t>(budget_bytes[i] / L.top_bytes, s.E)) : 0;
    L.cache_base = ctx->dev(off);
    off += align_up(L.top_bytes * L.slots, kAlign);
    L.slot_of.assign(s.E, -1);
    L.slot_owner.assign(L.slots, -1);
    for (hipEvent_t ev : L.pending_loads) ctx->free_events.push_back(ev);
    L.pending_loads.clear();
    L.has_pred = false;
    L.configured = true;
    if (top_slots_out) top_slots_out[i] = L.slots;
  }
  return MS_OK;
}

ms_status ms_load_top(ms_ctx* ctx, int32_t layer, int32_t e) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  LayerState& L = ctx->layers[layer];
  if (e < 0 || e >= ctx->s.E) return fail(ctx, MS_E_INVALID, "expert out of range");
  if (!L.configured) return fail(ctx, MS_E_STATE, "layer not configured");
  if (L.top_chunks == 0) return fail(ctx, MS_E_STATE, "layer split has no top segment");
  if (L.blob_of[e] < 0) return fail(ctx, MS_E_STATE, "expert weights not set");
  if (L.slot_of[e] >= 0) return fail(ctx, MS_E_STATE, "top segment already cached");
  int slot = -1;
  for (int i = 0; i < L.slots; ++i)
    if (L.slot_owner[i] < 0) {
      slot = i;
      break;
    }
  if (slot < 0) return fail(ctx, MS_E_BUDGET, "no free top-segment slot in this layer");
  if (L.has_last_fwd) {
    st = flush_fwd(ctx, L);
    if (st != MS_OK) return st;
    st = copy_after(ctx, L.last_fwd);
    if (st != MS_OK) return st;
  }
  st = issue_copy(ctx, L.cache_base + L.top_bytes * slot, ctx->blobs[L.blob_of[e]], ctx->blobs_dev[L.blob_of[e]],
                  L.top_bytes, MS_IV_COPY_TOP, layer);
  if (st != MS_OK) return st;
  hipEvent_t ev;
  MS_HIP(new_event(ctx, &ev));
  MS_HIP(hipEventRecord(ev, ctx->copy));
  L.pending_loads.push_back(ev);
  L.slot_of[e] = slot;
  L.slot_owner[slot] = e;
  return MS_OK;
}

ms_status ms_evict_top(ms_ctx* ctx, int32_t layer, int32_t e) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  LayerState& L = ctx->layers[layer];
  if (e < 0 || e >= ctx->s.E) return fail(ctx, MS_E_INVALID, "expert out of range");
  if (!L.configured || L.slot_of[e] < 0) return fail(ctx, MS_E_STATE, "top segment not cached");
  L.slot_owner[L.slot_of[e]] = -1;
  L.slot_of[e] = -1;
  return MS_OK;
}

ms_status ms_residency(ms_ctx* ctx, int32_t layer, uint8_t* state_out) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  if (!state_out) return fail(ctx, MS_E_INVALID, "state_out is NULL");
  const LayerState& L = ctx->layers[layer];
  for (int e = 0; e < ctx->s.E; ++e) {
    uint8_t v = 0;
    if (L.configured && L.slot_of[e] >= 0) v = (L.top_chunks >= ctx->s.n_chunks) ? 2 : 1;
    state_out[e] = v;
  }
  return MS_OK;
}

ms_status ms_drop_buffer(ms_ctx* ctx) {
  MS_CHECK_CTX(ctx);
  // groups already issued complete on the copy stream, which orders every
  // later copy into the same slots after them
  ctx->pf_queue.clear();
  ctx->pf_inflight.clear();
  for (BufSlot& b : ctx->buf) clear_slot(b);
  return MS_OK;
}

ms_status ms_prefetch(ms_ctx* ctx, int32_t layer, const int32_t* experts, int32_t n) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  if (n < 0 || (n > 0 && !experts)) return fail(ctx, MS_E_INVALID, "bad expert list");
  for (int i = 0; i < n; ++i)
    if (experts[i] < 0 || experts[i] >= ctx->s.E) return fail(ctx, MS_E_INVALID, "expert out of range");
  if (!ctx->layers[layer].configured) return fail(ctx, MS_E_STATE, "layer not configured");
  return enqueue_prefetch(ctx, layer, experts, n);
}

ms_status ms_predict(ms_ctx* ctx, int32_t layer, const void* h_dev, int32_t T, void* stream, int32_t* order_out,
                     float* score_out) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  const Shape& s = ctx->s;
  if (T < 1 || T > s.max_T || !h_dev || !order_out) return fail(ctx, MS_E_INVALID, "bad prediction arguments");
  if ((reinterpret_cast<uintptr_t>(h_dev) % 16) != 0) return fail(ctx, MS_E_INVALID, "h_dev not 16-byte aligned");
  LayerState& L = ctx->layers[layer];
  if (!L.router_set) return fail(ctx, MS_E_STATE, "router not set");
  hipStream_t sm = static_cast<hipStream_t>(stream);
  st = order_after_last(ctx, sm);
  if (st != MS_OK) return st;
  msk::LogitsArgs la{};
  la.h = h_dev;
  la.T = T;
  la.d = s.d;
  la.E = s.E;
  la.dtype = s.dtype;
  la.wr2 = ctx->dev(s.off_router + s.router_stride * layer);
  la.wt2 = ctx->dev(s.off_router_t + s.router_stride * layer);
  la.bias2 = L.bias_set ? reinterpret_cast<const float*>(ctx->dev(s.off_bias + s.bias_stride * layer)) : nullptr;
  la.logits2 = reinterpret_cast<float*>(ctx->dev(s.off_logits2));
  msk::RouteArgs rk{};
  rk.T = T;
  rk.E = s.E;
  rk.K = s.K;
  rk.renormalize = s.renorm;
  rk.logits_pred = la.logits2;
  set_route_workspace(ctx, &rk);
  rk.score = reinterpret_cast<float*>(ctx->dev(s.off_score));
  rk.order = reinterpret_cast<int32_t*>(ctx->dev(s.off_order));
  rk.host_score = ctx->d_score_map;
  rk.host_order = ctx->d_order_map;
  int ti = tl_begin(ctx, sm, MS_IV_PREDICT, layer, static_cast<uint64_t>(s.d) * s.E * s.elem);
  MS_HIP(msk::launch_logits_route(la, rk, sm));
  tl_end(ctx, ti, sm);
  MS_HIP(hipEventRecord(ctx->ev_last, sm));
  ctx->has_last = true;
  ctx->last_ev = ctx->ev_last;
  ctx->last_stream = sm;
  MS_HIP(hipEventSynchronize(ctx->ev_last));
  std::memcpy(order_out, const_cast<const int32_t*>(ctx->h_order), sizeof(int32_t) * s.E);
  if (score_out) std::memcpy(score_out, const_cast<const float*>(ctx->h_score), sizeof(float) * s.E);
  L.pred_order.assign(order_out, order_out + s.E);
  L.has_pred = true;
  return MS_OK;
}

ms_status ms_forward(ms_ctx* ctx, int32_t layer, const void* h_dev, int32_t T, float* y_dev, int32_t* idx_dev,
                     float* w_dev, int32_t flags, void* stream) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  const Shape& s = ctx->s;
  if (T < 0 || T > s.max_T) return fail(ctx, MS_E_INVALID, "T outside [0, max_tokens]");
  if (T == 0) return MS_OK;
  if (!h_dev || !y_dev || !idx_dev || !w_dev) return fail(ctx, MS_E_INVALID, "NULL device buffer");
  if ((reinterpret_cast<uintptr_t>(h_dev) % 16) != 0 || (reinterpret_cast<uintptr_t>(y_dev) % 16) != 0)
    return fail(ctx, MS_E_INVALID, "h_dev and y_dev must be 16-byte aligned");
  LayerState& L = ctx->layers[layer];
  if (!L.configured) return fail(ctx, MS_E_STATE, "layer not configured (ms_configure)");
  if (!L.router_set) return fail(ctx, MS_E_STATE, "router not set");
  for (int e = 0; e < s.E; ++e)
    if (L.blob_of[e] < 0) return fail(ctx, MS_E_STATE, "expert weights not set");
  for (int i = 0; i < s.n_sh; ++i)
    if (!L.shared_set[i]) return fail(ctx, MS_E_STATE, "shared expert weights not set");
  const bool predict_next = (flags & MS_FWD_PREDICT_NEXT) != 0;
  const int next_layer = (layer + 1) % s.L;
  if (predict_next && !ctx->layers[next_layer].router_set)
    return fail(ctx, MS_E_STATE, "next layer's router not set");

  hipStream_t sm = static_cast<hipStream_t>(stream);
  st = order_after_last(ctx, sm);
  if (st != MS_OK) return st;
  for (hipEvent_t ev : L.pending_loads) {
    MS_HIP(hipStreamWaitEvent(sm, ev, 0));
    ctx->free_events.push_back(ev);
  }
  L.pending_loads.clear();

  ctx->side_work = ctx->side2_work = false;
  const int TK = T * s.K;
  int32_t* d_offsets = reinterpret_cast<int32_t*>(ctx->dev(s.off_offsets));
  int32_t* d_perm = reinterpret_cast<int32_t*>(ctx->dev(s.off_perm));
  int32_t* d_pos = reinterpret_cast<int32_t*>(ctx->dev(s.off_pos));
  float* d_part = reinterpret_cast<float*>(ctx->dev(s.off_part));
  float* d_part_sh = reinterpret_cast<float*>(ctx->dev(s.off_part_sh));
  const int rows_routed = s.max_T * s.K;

  // 1. routing (+ next-layer prediction), grouping
  msk::LogitsArgs la{};
  la.h = h_dev;
  la.T = T;
  la.d = s.d;
  la.E = s.E;
  la.dtype = s.dtype;
  la.wr = ctx->dev(s.off_router + s.router_stride * layer);
  la.wt = ctx->dev(s.off_router_t + s.router_stride * layer);
  la.bias = L.bias_set ? reinterpret_cast<const float*>(ctx->dev(s.off_bias + s.bias_stride * layer)) : nullptr;
  la.logits = reinterpret_cast<float*>(ctx->dev(s.off_logits));
  if (predict_next) {
    const LayerState& N = ctx->layers[next_layer];
    la.wr2 = ctx->dev(s.off_router + s.router_stride * next_layer);
    la.wt2 = ctx->dev(s.off_router_t + s.router_stride * next_layer);
    la.bias2 = N.bias_set ? reinterpret_cast<const float*>(ctx->dev(s.off_bias + s.bias_stride * next_layer)) : nullptr;
    la.logits2 = reinterpret_cast<float*>(ctx->dev(s.off_logits2));
  }
  const uint64_t router_bytes = static_cast<uint64_t>(s.d) * s.E * s.elem * (predict_next ? 2 : 1);

  msk::RouteArgs ga{};
  ga.T = T;
  ga.E = s.E;
  ga.K = s.K;
  ga.renormalize = s.renorm;
  ga.logits = la.logits;
  ga.idx = idx_dev;
  ga.w = w_dev;
  ga.offsets = d_offsets;
  ga.perm = d_perm;
  ga.pos = d_pos;
  ga.host_offsets = ctx->d_offsets_map;
  ga.host_seq = ctx->d_seq_map;
  ga.seq = static_cast<int32_t>(++ctx->route_seq);
  set_route_workspace(ctx, &ga);
  if (predict_next) {
    ga.logits_pred = la.logits2;
    ga.score = reinterpret_cast<float*>(ctx->dev(s.off_score));
    ga.order = reinterpret_cast<int32_t*>(ctx->dev(s.off_order));
    ga.host_score = ctx->d_score_map;
    ga.host_order = ctx->d_order_map;
  }
  int ti = tl_begin(ctx, sm, MS_IV_ROUTER, layer, router_bytes);
  MS_HIP(msk::launch_logits_route(la, ga, sm));
  tl_end(ctx, ti, sm);
  // The host learns the routing from the completion word; side streams order
  // after it through ev_route, needed only when an expert misses chunks (a
  // marker between two kernels costs the stream a few microseconds).
  bool all_res = true;
  for (int e = 0; e < s.E && all_res; ++e) all_res = resident_chunks(L, e) >= s.n_chunks;
  if (!all_res) MS_HIP(hipEventRecord(ctx->ev_route, sm));

  // decode path (chunk kernel, launched before the host sees the routing)
  // or prefill path (matrix cores, launched once the token counts are known)
  bool prefill = s.dtype == MS_BF16 && static_cast<int64_t>(T) * s.K >= 8ll * s.E;
  if (flags & MS_FWD_MATRIX_CORES) prefill = s.dtype == MS_BF16;
  if (flags & MS_FWD_NO_MATRIX_CORES) prefill = false;
  // prefill: the resident experts' launches are planned on the device and
  // follow the routing at once (no host round trip)
  const bool planned = prefill && plan_on_device(s);
  int tl_pgu = -1, tl_pdn = -1;
  if (planned) {
    const ms_status pst = launch_planned(ctx, layer, h_dev, T, sm, &tl_pgu, &tl_pdn);
    if (pst != MS_OK) return pst;
  }

  // 2. segments already in VRAM (Eq. (5): processed while missing ones
  //    load): cached tops, staging-buffer groups of this layer whose copies
  //    have completed, and the shared experts.  Experts that turn out not to
  //    be selected exit at once.  (Decode path only.)
  msk::FfnArgs fa{};
  fa.h = h_dev;
  fa.offsets = d_offsets;
  fa.perm = d_perm;
  fa.part = d_part;
  fa.part_sh = d_part_sh;
  fa.chunk_bytes = s.chunk_bytes;
  fa.sh_plane = s.sh_plane;
  fa.rows_routed = rows_routed;
  fa.rows_shared = s.max_T;
  fa.d = s.d;
  fa.K = s.K;
  fa.T = T;
  fa.dtype = s.dtype;
  fa.subs = s.subs;
  fa.n_planes = s.n_chunks * s.subs;
  fa.n_planes_sh = s.n_chunks_sh * s.subs;
  fa.bits = s.bits;
  std::vector<msk::FfnTask> res_tasks;
  for (int e = 0; e < s.E && !prefill; ++e) {
    const int rc = resident_chunks(L, e);
    if (rc <= 0) continue;
    msk::FfnTask t{};
    t.base = L.cache_base + L.top_bytes * L.slot_of[e];
    t.expert = e;
    t.chunk_lo = 0;
    t.n_chunks = rc;
    res_tasks.push_back(t);
  }
  bool any_pre = false;
  for (BufSlot& b : ctx->buf) {
    if (b.layer != layer || prefill) continue;
    const int res = resident_chunks(L, b.expert);
    for (int gi = 0; gi < static_cast<int>(b.groups.size()); ++gi) {
      Group& g = b.groups[gi];
      const int lo = std::max(g.c_lo, res);
      if (!g.issued || lo >= g.c_hi) continue;
      const hipError_t q = group_landed(ctx, static_cast<int>(&b - ctx->buf.data()), gi);
      if (q == hipErrorNotReady) continue;
      if (q != hipSuccess) return poison(ctx, "hipEventQuery(group)", q);
      msk::FfnTask t{};
      t.base = b.base;
      t.expert = b.expert;
      t.chunk_lo = lo;
      t.n_chunks = g.c_hi - lo;
      if (!res_tasks.empty() && res_tasks.back().base == t.base && res_tasks.back().expert == t.expert &&
          res_tasks.back().chunk_lo + res_tasks.back().n_chunks == lo)
        res_tasks.back().n_chunks += t.n_chunks;  // contiguous with the previous group
      else
        res_tasks.push_back(t);
      g.pre = true;
      any_pre = true;
    }
  }
  auto shared_base = [&](int i) {
    return ctx->dev(s.off_shared + align_up(s.shared_bytes, kAlign) * (static_cast<uint64_t>(layer) * s.n_sh + i));
  };
  for (int i = 0; i < s.n_sh && !prefill; ++i) {
    msk::FfnTask t{};
    t.base = shared_base(i);
    t.expert = -1 - i;
    t.chunk_lo = 0;
    t.n_chunks = s.n_chunks_sh;
    res_tasks.push_back(t);
  }
  std::vector<int> res_tl;  // timeline records of resident launches (bytes fixed after routing)
  std::vector<std::vector<msk::FfnTask>> res_batches;
  auto launch_tasks = [&](const std::vector<msk::FfnTask>& tasks, hipStream_t st, int kind, int max_tok,
                          std::vector<int>* tl_ids, std::vector<std::vector<msk::FfnTask>>* batches) -> ms_status {
    for (size_t i0 = 0; i0 < tasks.size(); i0 += msk::kMaxTasks) {
      const size_t i1 = std::min(tasks.size(), i0 + msk::kMaxTasks);
      fa.n_tasks = static_cast<int>(i1 - i0);
      int wg = 0;
      uint64_t bytes = 0;
      for (size_t i = i0; i < i1; ++i) {
        fa.tasks[i - i0] = tasks[i];
        fa.tasks[i - i0].wg_begin = wg;
        wg += tasks[i].n_chunks * s.subs;
        bytes += s.chunk_bytes * tasks[i].n_chunks;
      }
      fa.n_wg = wg;
      const int id = tl_begin(ctx, st, kind, layer, bytes);
      MS_HIP(msk::launch_ffn(fa, max_tok, st));
      tl_end(ctx, id, st);
      if (tl_ids) tl_ids->push_back(id);
      if (batches) batches->emplace_back(tasks.begin() + i0, tasks.begin() + i1);
    }
    return MS_OK;
  };
  st = launch_tasks(res_tasks, sm, MS_IV_FFN_RESIDENT, T, &res_tl, &res_batches);
  if (st != MS_OK) return st;
  if (any_pre) MS_HIP(hipEventRecord(ctx->ev_res, sm));

  // 3. wait for the routing result on the host, keeping prefetch copies fed
  // (a launch that failed never sets the completion word: after a wait far
  // longer than a routing, the stream is checked every kRouteCheckMs; a
  // query puts a marker into the stream, which costs it microseconds)
  {
    auto next_check = std::chrono::steady_clock::now() + std::chrono::milliseconds(kRouteCheckMs);
    while (*reinterpret_cast<volatile int32_t*>(ctx->h_seq) != ga.seq) {
      if (std::chrono::steady_clock::now() >= next_check) {
        const hipError_t q = hipStreamQuery(sm);
        if (q != hipSuccess && q != hipErrorNotReady) return poison(ctx, "hipStreamQuery(route)", q);
        if (q == hipSuccess && *reinterpret_cast<volatile int32_t*>(ctx->h_seq) != ga.seq)
          return poison(ctx, "routing completion word", hipErrorLaunchFailure);
        next_check = std::chrono::steady_clock::now() + std::chrono::milliseconds(kRouteCheckMs);
      }
      st = pump_prefetch(ctx);
      if (st != MS_OK) return st;
    }
  }
  std::vector<int32_t> offs(s.E + 1);
  for (int e = 0; e <= s.E; ++e) offs[e] = reinterpret_cast<volatile int32_t*>(ctx->h_offsets)[e];
  std::vector<int> pred;
  if (predict_next) {
    pred.resize(s.E);
    for (int e = 0; e < s.E; ++e) pred[e] = reinterpret_cast<volatile int32_t*>(ctx->h_order)[e];
  }
  terminate_prefetch(ctx);
  ctx->pf_inflight.clear();  // in-flight groups complete on their own

  // bytes of the resident launches now that the active experts are known
  if (tl_pgu >= 0 || tl_pdn >= 0) {
    uint64_t gu = static_cast<uint64_t>(s.n_sh) * s.n_chunks_sh, dn = static_cast<uint64_t>(s.n_sh) * s.n_chunks_sh;
    for (int e = 0; e < s.E; ++e) {
      if (offs[e + 1] == offs[e]) continue;
      const int rc = resident_chunks(L, e);
      gu += rc;
      if (rc >= s.n_chunks) dn += s.n_chunks;
    }
    if (tl_pgu >= 0) ctx->tl[tl_pgu].bytes = gu * mma_gu_bytes(s);
    if (tl_pdn >= 0) ctx->tl[tl_pdn].bytes = dn * mma_dn_bytes(s);
  }
  for (size_t bi = 0; bi < res_tl.size(); ++bi) {
    if (res_tl[bi] < 0) continue;
    uint64_t bytes = 0;
    for (const msk::FfnTask& t : res_batches[bi]) {
      if (t.expert >= 0 && offs[t.expert + 1] == offs[t.expert]) continue;
      bytes += s.chunk_bytes * t.n_chunks;
    }
    ctx->tl[res_tl[bi]].bytes = bytes;
  }

  // 4. statistics of this routing (Sec. 3.4.1: alpha / beta / gamma; the
  //    configurator's H, P, PH and the cache priorities, Sec. 3.4.2)
  update_plan_stats(ctx, L, offs, T);
  L.st.forwards += 1;
  L.st.tokens += T;
  L.st.selected += TK;
  if (L.has_pred) {
    for (int k = 0; k < std::min<int>(s.K, static_cast<int>(L.pred_order.size())); ++k) {
      const int e = L.pred_order[k];
      if (offs[e + 1] > offs[e]) L.st.predicted_hits += 1;
    }
    L.st.predictions += 1;
    L.has_pred = false;
  }

  if (!prefill) {
  // 5. missing segments.  Side stream: first one wide launch over buffer
  //    groups that landed by now, then one launch per group still to land,
  //    each after its copy event.  Slots read by the resident launch are
  //    released only after it (the side stream waits for it).
  if (any_pre || !all_res) MS_HIP(hipStreamWaitEvent(ctx->side, any_pre ? ctx->ev_res : ctx->ev_route, 0));
  // slots already holding an active expert's missing part are reserved so
  // that no other miss of this forward evicts them first
  for (int e = 0; e < s.E; ++e) {
    if (offs[e + 1] == offs[e]) continue;
    const int si = find_slot(ctx, layer, e);
    if (si >= 0 && ctx->buf[si].first_chunk <= resident_chunks(L, e)) ctx->buf[si].use_order = kReserved;
  }
  int use_counter = 0;
  auto count_used = [&](Group& g) {
    if (g.prefetch && !g.used) L.st.bytes_prefetch_used += s.chunk_bytes * (g.c_hi - g.c_lo);
    g.used = true;
  };
  // 5a. landed groups of covering slots
  std::vector<msk::FfnTask> landed;
  std::vector<int> landed_slots;
  for (int e = 0; e < s.E; ++e) {
    if (offs[e + 1] == offs[e]) continue;
    const int res = resident_chunks(L, e);
    if (res >= s.n_chunks) continue;
    const int si = find_slot(ctx, layer, e);
    if (si < 0 || ctx->buf[si].first_chunk > res) continue;
    BufSlot& b = ctx->buf[si];
    bool any = false;
    for (int gi = 0; gi < static_cast<int>(b.groups.size()); ++gi) {
      Group& g = b.groups[gi];
      const int lo = std::max(g.c_lo, res);
      if (lo >= g.c_hi || !g.issued) continue;
      if (g.pre) {
        count_used(g);
        continue;
      }
      const hipError_t q = group_landed(ctx, si, gi);
      if (q == hipErrorNotReady) continue;
      if (q != hipSuccess) return poison(ctx, "hipEventQuery(group)", q);
      msk::FfnTask t{};
      t.base = b.base;
      t.expert = e;
      t.chunk_lo = lo;
      t.n_chunks = g.c_hi - lo;
      if (!landed.empty() && landed.back().base == t.base && landed.back().chunk_lo + landed.back().n_chunks == lo)
        landed.back().n_chunks += t.n_chunks;
      else
        landed.push_back(t);
      g.pre = true;  // computed now; the per-group pass skips it
      count_used(g);
      any = true;
    }
    if (any) landed_slots.push_back(si);
  }
  if (!landed.empty()) {
    ctx->side_work = true;
    st = launch_tasks(landed, ctx->side, MS_IV_FFN_STREAMED, T, nullptr, nullptr);
    if (st != MS_OK) return st;
  }
  for (BufSlot& b : ctx->buf) {
    bool read = false;
    for (const Group& g : b.groups) read = read || g.pre;
    if (read) {
      MS_HIP(hipEventRecord(b.last_read, ctx->side));
      b.has_last_read = true;
    }
  }
  // 5b. the rest: issue what is missing, compute each group as it lands
  for (int e = 0; e < s.E; ++e) {
    if (offs[e + 1] == offs[e]) continue;
    L.st.experts_active += 1;
    const int res = resident_chunks(L, e);
    if (res >= s.n_chunks)
      L.st.alpha += 1;
    else if (res > 0)
      L.st.beta += 1;
    else
      L.st.gamma += 1;
  }
  for (const int e : miss_order(ctx, layer, offs, nullptr)) {
    const int res = resident_chunks(L, e);
    int si = find_slot(ctx, layer, e);
    bool hit = false;
    if (si >= 0 && ctx->buf[si].first_chunk <= res) {
      for (const Group& g : ctx->buf[si].groups) hit = hit || g.issued;
    } else {
      if (si < 0) si = pick_victim(ctx, true);
      if (si < 0) return fail(ctx, MS_E_STATE, "no staging slot can be taken");
      st = assign_slot(ctx, si, layer, e, res, true);
      if (st != MS_OK) return st;
    }
    if (hit) L.st.buffer_hits += 1;
    BufSlot& b = ctx->buf[si];
    b.use_order = use_counter++;
    b.tick = ++ctx->tick;
    bool launched = false;
    for (int gi = 0; gi < static_cast<int>(b.groups.size()); ++gi) {
      Group& g = b.groups[gi];
      const int lo = std::max(g.c_lo, res);
      if (lo >= g.c_hi || g.pre) continue;
      if (!g.issued) {
        st = issue_group(ctx, si, gi, false);
        if (st != MS_OK) return st;
      }
      count_used(g);
      MS_HIP(hipStreamWaitEvent(ctx->side, b.gev[gi], 0));
      fa.n_tasks = 1;
      fa.tasks[0].base = b.base;
      fa.tasks[0].expert = static_cast<int16_t>(e);
      fa.tasks[0].chunk_lo = static_cast<uint16_t>(lo);
      fa.tasks[0].wg_begin = 0;
      fa.n_wg = (g.c_hi - lo) * s.subs;
      ctx->side_work = true;
      ti = tl_begin(ctx, ctx->side, MS_IV_FFN_STREAMED, layer, s.chunk_bytes * (g.c_hi - lo));
      MS_HIP(msk::launch_ffn(fa, offs[e + 1] - offs[e], ctx->side));
      tl_end(ctx, ti, ctx->side);
      launched = true;
    }
    if (launched) {
      MS_HIP(hipEventRecord(b.last_read, ctx->side));
      b.has_last_read = true;
    }
  }
  } else {
    st = prefill_experts(ctx, layer, h_dev, T, offs, sm, planned);
    if (st != MS_OK) return st;
  }
  for (BufSlot& b : ctx->buf)
    for (Group& g : b.groups) g.pre = false;
  // the combine needs the side stream only if this forward put kernels on
  // it (a cross-stream hand-off costs tens of microseconds)
  if (ctx->side_work) {
    MS_HIP(hipEventRecord(ctx->ev_side_done, ctx->side));
    MS_HIP(hipStreamWaitEvent(sm, ctx->ev_side_done, 0));
  }
  if (ctx->side2_work) {
    MS_HIP(hipEventRecord(ctx->ev_side2_done, ctx->side2));
    MS_HIP(hipStreamWaitEvent(sm, ctx->ev_side2_done, 0));
  }

  // 6. combine (Eq. (2) weighted sum, fixed order)
  msk::CombineArgs ca{};
  ca.part = d_part;
  ca.part_sh = d_part_sh;
  ca.pos = d_pos;
  ca.w = w_dev;
  ca.y = y_dev;
  ca.sh_plane = s.sh_plane;
  ca.rows_routed = rows_routed;
  ca.rows_shared = s.max_T;
  ca.n_planes = prefill ? s.down_splits : s.n_chunks * s.subs;
  ca.n_planes_sh = prefill ? 1 : s.n_chunks_sh * s.subs;
  ca.red = reinterpret_cast<float*>(ctx->dev(s.off_red));
  ca.pg = msk::combine_groups(T, s.K, s.n_sh, s.d, ca.n_planes);
  ca.n_shared = s.n_sh;
  ca.T = T;
  ca.K = s.K;
  ca.d = s.d;
  ti = tl_begin(ctx, sm, MS_IV_COMBINE, layer, 0);
  MS_HIP(msk::launch_combine(ca, sm));
  tl_end(ctx, ti, sm);

  // 6b. online replacement (Sec. 3.3): experts with no cached top that are
  //     now whole in a staging slot take the place of the lowest-ranked
  //     cached experts; the copies follow this forward's reads on `sm`
  if (ctx->policy != MS_CACHE_STATIC && L.slots > 0 && L.top_chunks > 0 && L.top_chunks <= s.n_chunks) {
    const std::vector<double> key = policy_key(ctx, L);
    std::vector<int> missed;
    for (int e = 0; e < s.E; ++e) {
      if (offs[e + 1] == offs[e] || L.slot_of[e] >= 0) continue;
      const int si = find_slot(ctx, layer, e);
      if (si >= 0 && ctx->buf[si].first_chunk == 0) missed.push_back(e);
    }
    std::stable_sort(missed.begin(), missed.end(), [&](int a, int b) { return key[a] > key[b]; });
    std::vector<char> fresh(s.E, 0);
    int inserted = 0;
    for (const int e : missed) {
      if (inserted >= L.slots) break;
      int slot = -1;
      for (int i = 0; i < L.slots && slot < 0; ++i)
        if (L.slot_owner[i] < 0) slot = i;
      if (slot < 0) {  // evict the lowest-ranked cached expert not cached just now
        int victim = -1;
        for (int i = 0; i < L.slots; ++i) {
          const int v = L.slot_owner[i];
          if (fresh[v]) continue;
          if (victim < 0 || key[v] < key[victim] || (key[v] == key[victim] && v < victim)) victim = v;
        }
        if (victim < 0) break;
        slot = L.slot_of[victim];
        L.slot_of[victim] = -1;
        L.slot_owner[slot] = -1;
      }
      BufSlot& b = ctx->buf[find_slot(ctx, layer, e)];
      const int cti = tl_begin(ctx, sm, MS_IV_COPY_TOP, layer, L.top_bytes);
      MS_HIP(msk::launch_d2d(L.cache_base + L.top_bytes * slot, b.base, L.top_bytes, sm));
      tl_end(ctx, cti, sm);
      MS_HIP(hipEventRecord(b.last_read, sm));
      b.has_last_read = true;
      L.slot_of[e] = slot;
      L.slot_owner[slot] = e;
      fresh[e] = 1;
      ++inserted;
      L.st.cache_inserts += 1;
    }
  }
  // the end of this forward, recorded when something waits for it
  L.fwd_unrecorded = true;
  L.fwd_stream = sm;
  L.has_last_fwd = true;
  ctx->has_last = true;
  ctx->last_ev = L.last_fwd;
  ctx->last_stream = sm;

  // 7. speculative prefetch of the next layer, predicted order (Sec. 3.2)
  if (predict_next) {
    LayerState& N = ctx->layers[next_layer];
    N.pred_order = pred;
    N.has_pred = true;
    if (N.configured) {
      // the paper's buffer holds K whole experts: prefetch candidates are the
      // K highest-ranked predictions, in rank order
      st = enqueue_prefetch(ctx, next_layer, pred.data(), std::min<int>(s.K, static_cast<int>(pred.size())));
      if (st != MS_OK) return st;
    }
  }
  for (BufSlot& b : ctx->buf) b.use_order = -1;
  return MS_OK;
}

ms_status ms_forward_noalloc(ms_ctx* ctx, int32_t layer, const void* h_dev, int32_t T, float* y_dev,
                             int32_t* idx_dev, float* w_dev, int32_t flags, void* stream) {
  MS_CHECK_CTX(ctx);
  const uint64_t need = ctx->s.off_buffer - ctx->s.off_logits;
  if (need > kStaticScratchBytes) {
    char msg[256];
    std::snprintf(msg, sizeof(msg),
                  "ms_forward_noalloc: this context's work buffers take %llu bytes, more than the %llu-byte static "
                  "scratch (lower max_tokens)",
                  static_cast<unsigned long long>(need), static_cast<unsigned long long>(kStaticScratchBytes));
    return fail(ctx, MS_E_UNSUPPORTED, msg);
  }
  if (!ctx->scratch_addr) return fail(ctx, MS_E_STATE, "ms_forward_noalloc: no static scratch on this device");
  ctx->work_base = ctx->scratch_addr;
  const ms_status st = ms_forward(ctx, layer, h_dev, T, y_dev, idx_dev, w_dev, flags, stream);
  ctx->work_base = nullptr;
  return st;
}

ms_status ms_residual_norm(ms_ctx* ctx, const void* h_dev, const float* y_dev, int32_t T, void* out_dev,
                           void* stream) {
  MS_CHECK_CTX(ctx);
  const Shape& s = ctx->s;
  if (T < 0 || T > s.max_T) return fail(ctx, MS_E_INVALID, "T outside [0, max_tokens]");
  if (T == 0) return MS_OK;
  if (!h_dev || !y_dev || !out_dev) return fail(ctx, MS_E_INVALID, "NULL device buffer");
  if ((reinterpret_cast<uintptr_t>(h_dev) | reinterpret_cast<uintptr_t>(y_dev) | reinterpret_cast<uintptr_t>(out_dev)) %
          16 != 0)
    return fail(ctx, MS_E_INVALID, "buffers must be 16-byte aligned");
  hipStream_t sm = static_cast<hipStream_t>(stream);
  ms_status st = order_after_last(ctx, sm);
  if (st != MS_OK) return st;
  MS_HIP(msk::launch_residual_norm(h_dev, y_dev, out_dev, T, s.d, s.dtype, 1e-6f, sm));
  return MS_OK;
}

ms_status ms_stats(ms_ctx* ctx, int32_t layer, ms_layer_stats* out) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  if (!out) return fail(ctx, MS_E_INVALID, "out is NULL");
  *out = ctx->layers[layer].st;
  return MS_OK;
}

ms_status ms_reset_stats(ms_ctx* ctx) {
  MS_CHECK_CTX(ctx);
  for (LayerState& L : ctx->layers) L.st = ms_layer_stats{};
  return MS_OK;
}

ms_status ms_plan_stats(ms_ctx* ctx, int32_t layer, double* hit, double* pred, double* pred_hit,
                        uint64_t* tokens_out) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  const LayerState& L = ctx->layers[layer];
  const int E = ctx->s.E;
  const uint64_t tot = L.q * static_cast<uint64_t>(ctx->s.K);
  if (hit) {
    uint64_t run = 0;
    hit[0] = 0.0;
    for (int c = 0; c < E; ++c) {
      run += L.hit_hist[c];
      hit[c + 1] = tot ? static_cast<double>(run) / static_cast<double>(tot) : 0.0;
    }
  }
  if (pred)
    for (int y = 0; y < E; ++y)
      pred[y] = L.q_pred ? static_cast<double>(L.pred_act[y]) / static_cast<double>(L.q_pred) : 0.0;
  if (pred_hit) {
    for (int y = 0; y < E; ++y) {
      double* row = pred_hit + static_cast<size_t>(y) * (E + 1);
      uint64_t run = 0;
      row[0] = 0.0;
      for (int c = 0; c < E; ++c) {
        run += L.pred_rank[static_cast<size_t>(y) * E + c];
        row[c + 1] = L.q_pred ? static_cast<double>(run) / static_cast<double>(L.q_pred) : 0.0;
      }
    }
  }
  if (tokens_out) {
    tokens_out[0] = L.q;
    tokens_out[1] = L.q_pred;
  }
  return MS_OK;
}

ms_status ms_reset_plan_stats(ms_ctx* ctx) {
  MS_CHECK_CTX(ctx);
  for (LayerState& L : ctx->layers) {
    std::fill(L.mu.begin(), L.mu.end(), 0.0);
    std::fill(L.nu.begin(), L.nu.end(), 0.0);
    std::fill(L.last_use.begin(), L.last_use.end(), 0);
    std::fill(L.hit_hist.begin(), L.hit_hist.end(), 0);
    std::fill(L.pred_act.begin(), L.pred_act.end(), 0);
    std::fill(L.pred_rank.begin(), L.pred_rank.end(), 0);
    L.clock = L.q = L.q_pred = 0;
  }
  return MS_OK;
}

ms_status ms_lcp_priority(ms_ctx* ctx, int32_t layer, double* prio_out) {
  MS_CHECK_CTX(ctx);
  ms_status st = check_layer(ctx, layer);
  if (st != MS_OK) return st;
  if (!prio_out) return fail(ctx, MS_E_INVALID, "prio_out is NULL");
  for (int e = 0; e < ctx->s.E; ++e) prio_out[e] = lcp_priority(ctx, ctx->layers[layer], e);
  return MS_OK;
}

ms_status ms_plan_solve(const ms_plan_problem* p, uint64_t v_e_bytes, double zeta, const uint64_t* start_budgets,
                        int32_t max_iter, uint64_t* budgets_out, double* theta_out, int32_t* cache_out,
                        double* exposed_us_out, int32_t* iters_out) {
  if (!p || !budgets_out || !p->hit || !p->pred || !p->pred_hit) return MS_E_INVALID;
  if (p->n_layers <= 0 || p->n_experts <= 0 || p->top_k <= 0 || p->top_k > p->n_experts || p->expert_bytes == 0 ||
      !(zeta > 0.0 && zeta < 1.0) || max_iter < 0 || v_e_bytes >= (1ull << 53) ||
      !(p->t_load_us >= 0.0) || !(p->t_moe_us >= 0.0) || !(p->t_att_us >= 0.0) || !(p->t_head_us >= 0.0))
    return MS_E_INVALID;
  msp::Problem pr{p->n_layers, p->n_experts, p->top_k, static_cast<double>(p->expert_bytes), p->t_att_us,
                  p->t_moe_us, p->t_head_us, p->t_load_us, p->hit, p->pred, p->pred_hit};
  std::vector<int64_t> V(p->n_layers);
  for (int i = 0; i < p->n_layers; ++i) {
    V[i] = start_budgets ? static_cast<int64_t>(start_budgets[i]) : static_cast<int64_t>(v_e_bytes / p->n_layers);
    if (V[i] <= 0) return MS_E_INVALID;
  }
  msp::Split out;
  const int it = msp::vram_allocation(pr, v_e_bytes, zeta, V, max_iter, &out);
  for (int i = 0; i < p->n_layers; ++i) {
    budgets_out[i] = static_cast<uint64_t>(V[i]);
    if (theta_out) theta_out[i] = out.theta[i];
    if (cache_out) cache_out[i] = out.C[i];
    if (exposed_us_out) exposed_us_out[i] = out.exposed[i];
  }
  if (iters_out) *iters_out = it;
  return MS_OK;
}

ms_status ms_cache_update(ms_ctx* ctx, const uint64_t* budgets, const float* r) {
  MS_CHECK_CTX(ctx);
  std::vector<int32_t> slots(ctx->s.L);
  ms_status st = ms_configure(ctx, budgets, r, slots.data());
  if (st != MS_OK) return st;
  for (int l = 0; l < ctx->s.L; ++l) {
    const std::vector<int> order = priority_order(ctx, ctx->layers[l]);
    for (int c = 0; c < slots[l]; ++c) {
      if (ctx->layers[l].blob_of[order[c]] < 0) continue;
      st = ms_load_top(ctx, l, order[c]);
      if (st != MS_OK) return st;
    }
  }
  return MS_OK;
}

ms_status ms_set_cache_policy(ms_ctx* ctx, int32_t policy, double rho, double omega, uint64_t seed) {
  MS_CHECK_CTX(ctx);
  if (policy < MS_CACHE_STATIC || policy > MS_CACHE_RND) return fail(ctx, MS_E_INVALID, "unknown cache policy");
  if (!(rho > 0.0 && rho < 1.0) || !(omega > 0.0)) return fail(ctx, MS_E_INVALID, "rho must be in (0, 1), omega > 0");
  ctx->policy = policy;
  ctx->rho = rho;
  ctx->omega = omega;
  ctx->rng = seed ^ 0x9e3779b97f4a7c15ull;
  return MS_OK;
}

ms_status ms_set_copy_engine(ms_ctx* ctx, int32_t engine) {
  MS_CHECK_CTX(ctx);
  if (engine != MS_COPY_KERNEL && engine != MS_COPY_DMA) return fail(ctx, MS_E_INVALID, "unknown copy engine");
  if (engine == MS_COPY_DMA && !ctx->dma_warm) {
    // the first DMA transfer of a process takes milliseconds (copies under
    // 64 KiB do not absorb that): pay it here, into the partials workspace,
    // which holds nothing between forwards
    constexpr uint64_t kWarmBytes = 1ull << 20;
    const uint64_t n = std::min<uint64_t>(kWarmBytes, ctx->s.part_bytes);
    void* hp = nullptr;
    if (n > 0 && hipHostMalloc(&hp, n, hipHostMallocDefault) == hipSuccess && hp) {
      std::memset(hp, 0, n);
      ms_status st = ms_sync(ctx);
      if (st == MS_OK) {
        hipError_t e = hipMemcpyAsync(ctx->dev(ctx->s.off_part), hp, n, hipMemcpyHostToDevice, ctx->copy);
        if (e == hipSuccess) e = hipStreamSynchronize(ctx->copy);
        if (e != hipSuccess) st = poison(ctx, "DMA warm-up copy", e);
      }
      (void)hipHostFree(hp);
      if (st != MS_OK) return st;
      ctx->dma_warm = true;
    } else {
      (void)hipGetLastError();
      return fail(ctx, MS_E_NOMEM, "pinned buffer for the DMA warm-up copy");
    }
  }
  ctx->copy_engine = engine;
  return MS_OK;
}

ms_status ms_timeline_begin(ms_ctx* ctx, void* stream, int32_t capacity) {
  MS_CHECK_CTX(ctx);
  if (capacity <= 0) return fail(ctx, MS_E_INVALID, "capacity must be positive");
  if (ctx->tl_on) return fail(ctx, MS_E_STATE, "timeline already running");
  for (TlRec& r : ctx->tl) {
    ctx->tl_pool.push_back(r.e0);
    ctx->tl_pool.push_back(r.e1);
  }
  ctx->tl.clear();
  // every record's two events exist before recording starts: creating
  // events while work is in flight would perturb what is measured
  while (static_cast<int64_t>(ctx->tl_pool.size()) < 2ll * capacity) {
    hipEvent_t ev;
    MS_HIP(hipEventCreate(&ev));
    ctx->tl_pool.push_back(ev);
  }
  if (!ctx->tl_origin) MS_HIP(hipEventCreate(&ctx->tl_origin));
  MS_HIP(hipEventRecord(ctx->tl_origin, static_cast<hipStream_t>(stream)));
  ctx->tl_on = true;
  ctx->tl_cap = capacity;
  return MS_OK;
}

ms_status ms_timeline_end(ms_ctx* ctx, ms_interval* out, int32_t cap, int32_t* n_out) {
  MS_CHECK_CTX(ctx);
  if (!ctx->tl_on) return fail(ctx, MS_E_STATE, "timeline not running");
  ms_status st = ms_sync(ctx);
  if (st != MS_OK) return st;
  MS_HIP(hipEventSynchronize(ctx->tl_origin));
  int n = 0;
  for (const TlRec& r : ctx->tl) {
    MS_HIP(hipEventSynchronize(r.e1));
    if (out && n < cap) {
      float a = 0.f, b = 0.f;
      MS_HIP(hipEventElapsedTime(&a, ctx->tl_origin, r.e0));
      MS_HIP(hipEventElapsedTime(&b, ctx->tl_origin, r.e1));
      out[n].kind = r.kind;
      out[n].layer = r.layer;
      out[n].t0_ms = a;
      out[n].t1_ms = b;
      out[n].bytes = r.bytes;
      ++n;
    }
  }
  if (n_out) *n_out = n;
  ctx->tl_on = false;
  return MS_OK;
}

}  // extern "C"
