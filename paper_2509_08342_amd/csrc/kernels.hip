// kernels.hip -- gfx950 kernels of libmoesplit: router + top-K (+ next-layer
// prediction), token grouping, prediction ranking, segment-aware SwiGLU over
// weight chunks, and the fixed-order combine.
//
// Paper: arXiv 2509.08342.  Router/top-K and the weighted expert sum follow
// Sec. 2.1 Eq. (2); the prediction follows Sec. 3.2 Eq. (3); the SwiGLU
// kernel computes one 64-unit chunk of an expert's FFN intermediate axis, so
// the same code runs on resident top-segment chunks and on streamed
// bottom-segment chunks (Sec. 3.1: segments are combined at compute time).
#include <hip/hip_runtime.h>
#include <math.h>

#include <algorithm>
#include <stdint.h>

#include "kernels.h"

namespace msk {

// ------------------------------------------------------------------ helpers

__device__ __forceinline__ float bf16f(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(uint16_t x) { return bf16f(x); }

template <typename W>
struct Vec;
template <>
struct Vec<float> {
  static constexpr int N = 4;
};
template <>
struct Vec<uint16_t> {
  static constexpr int N = 8;
};

// 16-byte load of weights or activations, widened to fp32.
__device__ __forceinline__ void load16(const float* p, float (&o)[4]) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  o[0] = v.x;
  o[1] = v.y;
  o[2] = v.z;
  o[3] = v.w;
}
__device__ __forceinline__ void load16(const uint16_t* p, float (&o)[8]) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  o[0] = __uint_as_float(v.x << 16);
  o[1] = __uint_as_float(v.x & 0xffff0000u);
  o[2] = __uint_as_float(v.y << 16);
  o[3] = __uint_as_float(v.y & 0xffff0000u);
  o[4] = __uint_as_float(v.z << 16);
  o[5] = __uint_as_float(v.z & 0xffff0000u);
  o[6] = __uint_as_float(v.w << 16);
  o[7] = __uint_as_float(v.w & 0xffff0000u);
}

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// 16-byte load of expert weights, which are streamed once per forward.
__device__ __forceinline__ uint4 ldw16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ void unpack(const uint4 v, float (&o)[4]) {
  o[0] = __uint_as_float(v.x);
  o[1] = __uint_as_float(v.y);
  o[2] = __uint_as_float(v.z);
  o[3] = __uint_as_float(v.w);
}
__device__ __forceinline__ void unpack(const uint4 v, float (&o)[8]) {
  o[0] = __uint_as_float(v.x << 16);
  o[1] = __uint_as_float(v.x & 0xffff0000u);
  o[2] = __uint_as_float(v.y << 16);
  o[3] = __uint_as_float(v.y & 0xffff0000u);
  o[4] = __uint_as_float(v.z << 16);
  o[5] = __uint_as_float(v.z & 0xffff0000u);
  o[6] = __uint_as_float(v.w << 16);
  o[7] = __uint_as_float(v.w & 0xffff0000u);
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// v_mfma_f32_16x16x32_bf16: lane l holds A[row l%16][8 k from 8*(l/16)],
// B[8 k from 8*(l/16)][column l%16] and the result C[rows 4*(l/16)+r][column
// l%16].  The k order inside a step is the same for A and B, which is all
// the contraction needs.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

__device__ __forceinline__ f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// -------------------------------------------------------------------- route
//
// Per token (one wave): K rounds of wave argmax over the untaken experts
// (larger logit wins, the lower index on equal logits; a NaN logit reads as
// -inf here and in the softmax scores), then
// the Eq. (2) weights from exp(logit - max).  Per token for the prediction
// (Sec. 3.2, Eq. (3)): the softmax of its second logits, added to the
// lane's running expert sums.  The grouping is a stable counting sort of
// the T*K slots by expert.  The prediction ranking orders experts by
// descending summed score, the lower index first on equal scores.

// Expert values per lane of a launch (QN = ceil(E / 64), a power of two):
// the routing kernels exist for QN = 1, 2, 4 and 8, so that a lane loops over
// its real experts only.  Lanes past E hold -inf and add nothing, so QN
// changes no result.
__host__ __device__ constexpr int lanes_q(int E) { return E <= 64 ? 1 : E <= 128 ? 2 : E <= 256 ? 4 : 8; }
static_assert(kMaxExperts <= 64 * 8, "at most 8 expert values per lane");

// Wave-wide reductions whose result does not depend on the order of the
// combination (max of floats, unsigned max) move data with DPP inside rows
// of 16 lanes -- lane i with i ^ 1, i ^ 2 (quad permutes), i ^ 7 (half-row
// mirror), i ^ 15 (row mirror) -- and read the four row results with
// v_readlane, instead of six LDS-crossbar permutes.  Floating-point sums
// keep their fixed butterflies.
constexpr int kDppXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror
constexpr int kDppMirror = 0x140;      // row_mirror

template <int CTRL>
__device__ __forceinline__ int dpp_move(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_move(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ int lane_read(int x, int l) { return __builtin_amdgcn_readlane(x, l); }
__device__ __forceinline__ float lane_read(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_move<kDppXor1>(v));
  v = fmaxf(v, dpp_move<kDppXor2>(v));
  v = fmaxf(v, dpp_move<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_move<kDppMirror>(v));
  return fmaxf(fmaxf(lane_read(v, 0), lane_read(v, 16)), fmaxf(lane_read(v, 32), lane_read(v, 48)));
}
__device__ __forceinline__ uint32_t wave_umax(uint32_t v) {
  v = max(v, static_cast<uint32_t>(dpp_move<kDppXor1>(static_cast<int>(v))));
  v = max(v, static_cast<uint32_t>(dpp_move<kDppXor2>(static_cast<int>(v))));
  v = max(v, static_cast<uint32_t>(dpp_move<kDppHalfMirror>(static_cast<int>(v))));
  v = max(v, static_cast<uint32_t>(dpp_move<kDppMirror>(static_cast<int>(v))));
  const uint32_t a = static_cast<uint32_t>(lane_read(static_cast<int>(v), 0));
  const uint32_t b = static_cast<uint32_t>(lane_read(static_cast<int>(v), 16));
  const uint32_t c = static_cast<uint32_t>(lane_read(static_cast<int>(v), 32));
  const uint32_t d = static_cast<uint32_t>(lane_read(static_cast<int>(v), 48));
  return max(max(a, b), max(c, d));
}

// Order-preserving integer image of a non-NaN float (-0 reads as +0, so
// equal floats have equal keys), and back.
__device__ __forceinline__ uint32_t float_key(float v) {
  const uint32_t b = __float_as_uint(v == 0.0f ? 0.0f : v);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// The logits of one token: lane l holds experts l + 64 q (-inf past E).
template <int QN>
__device__ __forceinline__ void load_lanes(const float* lg, int E, int lane, float (&lv)[QN]) {
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int e = lane + 64 * q;
    lv[q] = e < E ? lg[e] : -INFINITY;
  }
}

// Selection of one token by one wave from its logits (load_lanes); lanes
// k < K return the k-th pick and its weight.  A round takes the wave's
// largest untaken logit (an unsigned max over the lanes of the logits'
// order-preserving keys; untaken experts only, the others read as key 0,
// below every logit's) and then the lowest expert index holding it
// (ballots), which is the argmax with the lower index first on equal
// logits; the exponentials of the picks and their sum (in pick order)
// follow the rounds.
template <int QN>
__device__ __forceinline__ void select_token(const float (&lg)[QN], int E, int K, int renormalize, int lane,
                                             int& my_idx, float& my_w) {
  float lv[QN];
  uint32_t kv[QN];
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    float v = lg[q];
    if (v != v) v = -INFINITY;  // NaN reads as -inf, so an index is always found
    lv[q] = v;
    kv[q] = float_key(v);  // >= key(-inf) > 0
  }
  uint32_t open = 0;  // bit q: expert lane + 64 q exists and is not taken
#pragma unroll
  for (int q = 0; q < QN; ++q) open |= (lane + 64 * q < E ? 1u : 0u) << q;
  uint32_t mk = 0, my_k = 0;
  my_idx = 0;
  for (int k = 0; k < K; ++k) {
    uint32_t c = 0;
#pragma unroll
    for (int q = 0; q < QN; ++q) c = max(c, ((open >> q) & 1u) ? kv[q] : 0u);
    const uint32_t bk = wave_umax(c);
    int bi = 0;
    bool found = false;
#pragma unroll
    for (int q = 0; q < QN; ++q) {
      const uint64_t hit = __ballot(((open >> q) & 1u) && kv[q] == bk);
      if (!found && hit != 0) {
        bi = 64 * q + __ffsll(static_cast<unsigned long long>(hit)) - 1;
        found = true;
      }
    }
    if ((bi & 63) == lane) open &= ~(1u << (bi >> 6));
    if (k == 0) mk = bk;  // the first pick is the largest logit
    if (lane == k) {
      my_k = bk;
      my_idx = bi;
    }
  }
  const float m = key_float(mk);
  const float my_ex = lane < K ? expf(key_float(my_k) - m) : 0.0f;
  float zsel = 0.0f;
  for (int k = 0; k < K; ++k) zsel += lane_read(my_ex, k);
  float z = zsel;
  if (!renormalize) {
    float part = 0.0f;
#pragma unroll
    for (int q = 0; q < QN; ++q)
      if (lane + 64 * q < E) part += expf(lv[q] - m);
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) part += __shfl_xor(part, s, 64);
    z = part;
  }
  my_w = my_ex / z;
}

// acc[q] (expert lane + 64 q) += softmax(lg)[expert], one token's second
// logits (load_lanes), one wave.
template <int QN>
__device__ __forceinline__ void pred_add(const float (&lg)[QN], int E, int lane, float (&acc)[QN]) {
  float lv[QN];
  float m = -INFINITY;
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int e = lane + 64 * q;
    float v = e < E ? lg[q] : -INFINITY;
    if (v != v) v = -INFINITY;  // a NaN logit reads as -inf: score 0
    lv[q] = v;
    m = fmaxf(m, lv[q]);
  }
  m = wave_max(m);
  float z = 0.0f;
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    lv[q] = (lane + 64 * q < E) ? expf(lv[q] - m) : 0.0f;
    z += lv[q];
  }
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) z += __shfl_xor(z, s, 64);
#pragma unroll
  for (int q = 0; q < QN; ++q) acc[q] += lv[q] / z;
}

// Ranks of E scores: rank(e) = #{o : s_o > s_e, or s_o == s_e and o < e},
// so equal scores keep the lower index first.  rank_key(s_e, e) packs the
// order-preserving integer image of the float (the float order for every
// non-NaN score, and a strict total order whatever the values, so the ranks
// always form a permutation) above ~e, and rank(e) = #{o : key_o > key_e}.
// The E x E comparisons are shared by the NT threads of the work-group:
// thread (e, part) counts one part of the o range and adds its count to
// rank_s[e] (LDS, zero before the call).
__device__ __forceinline__ uint64_t rank_key(float v, int e) {
  const uint32_t b = __float_as_uint(v);
  const uint32_t k = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return (static_cast<uint64_t>(k) << 32) | static_cast<uint32_t>(~e);
}
__device__ __forceinline__ void rank_count(const uint64_t* key_s, int* rank_s, int E, int tid, int NT) {
  const int parts = max(1, NT / E);
  const int per = (E + parts - 1) / parts;
  if (tid < 0 || tid >= E * parts) return;
  const int e = tid % E, part = tid / E;
  const uint64_t v = key_s[e];
  const int o0 = part * per, o1 = min(E, o0 + per);
  int r = 0;
#pragma unroll 4
  for (int o = o0; o < o1; ++o) r += key_s[o] > v;
  if (r != 0) atomicAdd(&rank_s[e], r);
}

// Exclusive scan of cnt[0..E) by wave 0 into offs[0..E] (LDS); base (LDS,
// optional) receives the same values.
__device__ __forceinline__ void scan_offsets(const int* cnt, int* base, int* offs, int E, int lane) {
  int run = 0;
  for (int e0 = 0; e0 < E; e0 += 64) {
    const int e = e0 + lane;
    const int c = e < E ? cnt[e] : 0;
    int incl = c;
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) {
      const int o = __shfl_up(incl, s, 64);
      if (lane >= s) incl += o;
    }
    if (e < E) {
      if (base) base[e] = run + incl - c;
      offs[e] = run + incl - c;
    }
    run += lane_read(incl, 63);
  }
  if (lane == 0) offs[E] = run;
}

// The host-visible copies of the routing, all written by one wave (wave 0)
// so that one system-scope fence of that wave orders every copy before the
// completion word: host_rows as soon as the offsets and the prediction
// scores are known (their writes cross the bus while the work-group goes
// on), host_publish with the prediction order at the end, then the fence and
// the word.  Whole rows of consecutive values, so they cross the bus as few
// large writes.
__device__ __forceinline__ void host_rows(const RouteArgs& a, const int* offs_s, const float* score_s, int lane) {
  if (a.host_offsets != nullptr && offs_s != nullptr)
    for (int e = lane; e <= a.E; e += 64) a.host_offsets[e] = offs_s[e];
  if (a.host_score != nullptr && score_s != nullptr)
    for (int i = lane; i < a.E; i += 64) a.host_score[i] = score_s[i];
}
__device__ __forceinline__ void host_publish(const RouteArgs& a, const int* order_s, int lane) {
  if (a.host_order != nullptr && order_s != nullptr)
    for (int i = lane; i < a.E; i += 64) a.host_order[i] = order_s[i];
  if (a.host_offsets != nullptr || a.host_order != nullptr || a.host_score != nullptr || a.host_seq != nullptr)
    __threadfence_system();
  if (a.host_seq != nullptr && lane == 0) *reinterpret_cast<volatile int32_t*>(a.host_seq) = a.seq;
}

// Few tokens (T * K <= kFewSlots <= 64 NW, so one slot per thread):
// everything after the logits in one work-group of NW waves, in four
// barrier-separated steps --
//   1. per token, one wave: its selection, and its softmax of the second
//      logits added to the wave's running expert sums (prediction);
//   2. per wave: each of its 64 slots' rank among the wave's earlier slots of
//      the same expert, and the wave's count of each expert; the prediction
//      scores, summed over the waves in order;
//   3. wave 0: expert totals and their exclusive scan (offsets); the other
//      waves: the ranks of the prediction scores;
//   4. slot s goes to offsets[e] + (earlier waves' slots of e) + (its rank
//      in its wave), a stable counting sort; expert e goes to position
//      rank(e) of the prediction order.
// Every result stays in LDS until the last barrier and is then stored once
// (a barrier after a store to memory would wait for it).
constexpr int kFewSlots = 1024;

// The route body's LDS.
template <int NW>
struct RouteLds {
  uint64_t key_s[kMaxExperts];
  int idx_s[kFewSlots];
  float w_s[kFewSlots];
  int perm_s[kFewSlots];
  int pos_s[kFewSlots];
  int offs_s[kMaxExperts + 1];
  int cnt_s[kMaxExperts];
  float score_s[kMaxExperts];
  int rank_s[kMaxExperts];
  int order_s[kMaxExperts];
  int wcnt[NW][kMaxExperts];    // per-wave slot counts
  float wsum[NW][kMaxExperts];  // per-wave prediction sums
};

template <int NW, int QN>
__device__ void route_body(const RouteArgs& a, RouteLds<NW>& L) {
  static_assert(kFewSlots <= 64 * NW, "one slot per thread");
  int* idx_s = L.idx_s;
  float* w_s = L.w_s;
  int* perm_s = L.perm_s;
  int* pos_s = L.pos_s;
  int* offs_s = L.offs_s;
  int* cnt_s = L.cnt_s;
  float* score_s = L.score_s;
  uint64_t* key_s = L.key_s;
  int* rank_s = L.rank_s;
  int* order_s = L.order_s;
  auto& wcnt = L.wcnt;
  auto& wsum = L.wsum;
  constexpr int NT = 64 * NW;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int E = a.E, K = a.K;
  const int TK = a.T * K;
  const bool sel = a.logits != nullptr, pred = a.logits_pred != nullptr;

  // counts and ranks start at zero (each wave clears its own row of counts;
  // all are first read after the next barrier)
  for (int e = lane; e < E; e += 64) wcnt[wave][e] = 0;
  for (int e = tid; e < E; e += NT) rank_s[e] = 0;

  // 1. selection and prediction sums, one wave per token; both rows of a
  //    token are requested together (one memory round trip)
  float acc[QN];
#pragma unroll
  for (int q = 0; q < QN; ++q) acc[q] = 0.0f;
  for (int t = wave; t < a.T; t += NW) {
    float lg[QN], lp[QN];
    if (sel) load_lanes(a.logits + static_cast<size_t>(t) * E, E, lane, lg);
    if (pred) load_lanes(a.logits_pred + static_cast<size_t>(t) * E, E, lane, lp);
    if (sel) {
      int my_idx;
      float my_w;
      select_token(lg, E, K, a.renormalize, lane, my_idx, my_w);
      if (lane < K) {
        idx_s[t * K + lane] = my_idx;
        w_s[t * K + lane] = my_w;
      }
    }
    if (pred) pred_add(lp, E, lane, acc);
  }
  if (pred) {
#pragma unroll
    for (int q = 0; q < QN; ++q)
      if (lane + 64 * q < E) wsum[wave][lane + 64 * q] = acc[q];
  }
  __syncthreads();

  // 2. per-wave slot ranks and counts; prediction scores
  int ge = -1, grank = 0;
  if (sel) {
    // indices lie in [0, E) (selection above); the clamp only keeps LDS
    // accesses in bounds whatever the input
    ge = tid < TK ? min(max(idx_s[tid], 0), E - 1) : -1;
    const int s0 = wave * 64, s1 = min(TK, s0 + 64);
    if (s0 < s1) {
      const int t_first = s0 / K, t_last = (s1 - 1) / K;
      if (t_last - t_first < E) {
        // the wave's tokens in order: the slots of one token (distinct
        // experts) take the running count of their expert as their rank and
        // add one, so the counts end as the wave's counts
        const int my_t = tid / K;
        for (int t = t_first; t <= t_last; ++t)
          if (my_t == t && ge >= 0) grank = atomicAdd(&wcnt[wave][ge], 1);
      } else {
        // more tokens than experts in the wave: one ballot per distinct
        // expert instead (the same ranks and counts)
        const uint64_t lt = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
        uint64_t pending = __ballot(ge >= 0);
        while (pending) {
          const int leader = __ffsll(static_cast<unsigned long long>(pending)) - 1;
          const int le = lane_read(ge, leader);
          const uint64_t same = __ballot(ge == le);
          if (ge == le) grank = __popcll(same & lt);
          if (lane == leader) wcnt[wave][le] = __popcll(same);
          pending &= ~same;
        }
      }
    }
  }
  if (pred) {
    for (int e = tid; e < E; e += NT) {
      float sc = 0.0f;
      for (int w2 = 0; w2 < NW; ++w2) sc += wsum[w2][e];
      score_s[e] = sc;
      key_s[e] = rank_key(sc, e);
    }
  }
  __syncthreads();

  // 3. offsets and the first host-visible copies (wave 0); prediction ranks
  //    (the other waves when wave 0 has the offsets to do)
  if (wave == 0) {
    if (sel) {
      for (int e = lane; e < E; e += 64) {
        int c = 0;
        for (int w2 = 0; w2 < NW; ++w2) c += wcnt[w2][e];
        cnt_s[e] = c;
      }
      scan_offsets(cnt_s, nullptr, offs_s, E, lane);
    }
    host_rows(a, sel ? offs_s : nullptr, pred ? score_s : nullptr, lane);
  }
  if (pred) rank_count(key_s, rank_s, E, sel ? tid - 64 : tid, sel ? NT - 64 : NT);
  __syncthreads();

  // 4. grouped positions; prediction order
  if (ge >= 0) {
    int p = offs_s[ge] + grank;
    for (int w2 = 0; w2 < wave; ++w2) p += wcnt[w2][ge];
    perm_s[p] = tid;
    pos_s[tid] = p;
  }
  if (pred)
    for (int e = tid; e < E; e += NT) order_s[rank_s[e]] = e;
  __syncthreads();

  // the results to memory, then their host-visible copies
  if (sel) {
    for (int i = tid; i < TK; i += NT) {
      a.idx[i] = idx_s[i];
      a.w[i] = w_s[i];
      a.perm[i] = perm_s[i];
      a.pos[i] = pos_s[i];
    }
    for (int e = tid; e <= E; e += NT) a.offsets[e] = offs_s[e];
  }
  if (pred) {
    for (int i = tid; i < E; i += NT) {
      a.order[i] = order_s[i];
      a.score[i] = score_s[i];
    }
  }
  if (wave == 0) host_publish(a, pred ? order_s : nullptr, lane);
}

constexpr int kRouteWaves = 16;

template <int QN>
__global__ __launch_bounds__(64 * kRouteWaves) void route_kernel(RouteArgs a) {
  __shared__ RouteLds<kRouteWaves> lds;
  route_body<kRouteWaves, QN>(a, lds);
}

// Many tokens, step 1 (work-group b: tokens [b TB, (b+1) TB), one wave per
// token): selection, then each slot's rank among the block's earlier slots
// of the same expert and the block's expert counts blk[e][b]; the block's
// prediction score sums (waves in order) into psc[e][b].
constexpr int kSelWaves = 16;  // one wave per token of a block of at most 16

template <int QN>
__global__ __launch_bounds__(64 * kSelWaves) void select_many_kernel(RouteArgs a, int TB) {
  __shared__ int sidx[64 * kSelWaves];
  __shared__ int cnt[kMaxExperts];
  __shared__ float wsc[kSelWaves][kMaxExperts];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int E = a.E, K = a.K;
  const int b = blockIdx.x, t0 = b * TB, t1 = min(a.T, t0 + TB);
  if (a.logits != nullptr) {
    for (int e = tid; e < E; e += 64 * kSelWaves) cnt[e] = 0;
    for (int t = t0 + wave; t < t1; t += kSelWaves) {
      int my_idx;
      float my_w;
      float lg[QN];
      load_lanes(a.logits + static_cast<size_t>(t) * E, E, lane, lg);
      select_token(lg, E, K, a.renormalize, lane, my_idx, my_w);
      if (lane < K) {
        a.idx[static_cast<size_t>(t) * K + lane] = my_idx;
        a.w[static_cast<size_t>(t) * K + lane] = my_w;
        sidx[(t - t0) * K + lane] = my_idx;
      }
    }
    __syncthreads();
    const int n = (t1 - t0) * K;  // <= TB * K <= 64 * kSelWaves
    if (tid < n) {
      const int e = min(max(sidx[tid], 0), E - 1);
      int r = 0;
      for (int j = 0; j < tid; ++j) r += (sidx[j] == e);
      a.lrank[static_cast<size_t>(t0) * K + tid] = r;
      atomicAdd(&cnt[e], 1);
    }
    __syncthreads();
    for (int e = tid; e < E; e += 64 * kSelWaves) a.blk[static_cast<size_t>(e) * a.nblk_cap + b] = cnt[e];
  }
  if (a.logits_pred != nullptr) {
    float acc[QN];
#pragma unroll
    for (int q = 0; q < QN; ++q) acc[q] = 0.0f;
    for (int t = t0 + wave; t < t1; t += kSelWaves) {
      float lp[QN];
      load_lanes(a.logits_pred + static_cast<size_t>(t) * E, E, lane, lp);
      pred_add(lp, E, lane, acc);
    }
#pragma unroll
    for (int q = 0; q < QN; ++q)
      if (lane + 64 * q < E) wsc[wave][lane + 64 * q] = acc[q];
    __syncthreads();
    for (int e = tid; e < E; e += 64 * kSelWaves) {
      float sc = wsc[0][e];
#pragma unroll
      for (int w2 = 1; w2 < kSelWaves; ++w2) sc += wsc[w2][e];
      a.psc[static_cast<size_t>(e) * a.nblk_cap + b] = sc;
    }
  }
}

// Many tokens, step 2 (one work-group): per expert the exclusive prefix of
// its block counts (in place in blk) and its total; the exclusive scan over
// experts into offsets; the prediction scores summed over blocks in order,
// and their ranking.
constexpr int kScanWaves = 16;
constexpr int kScanGroup = 8;  // experts per wave whose loads are in flight together

__global__ __launch_bounds__(64 * kScanWaves) void scan_many_kernel(RouteArgs a, int nblk) {
  __shared__ int tot[kMaxExperts];
  __shared__ int offs_s[kMaxExperts + 1];
  __shared__ float score_s[kMaxExperts];
  __shared__ uint64_t key_s[kMaxExperts];
  __shared__ int rank_s[kMaxExperts];
  __shared__ int order_s[kMaxExperts];
  // a wave takes kScanGroup experts at a time (e0, e0 + kScanWaves, ...) and
  // requests their values of 64 blocks together, so that the experts of a
  // wave cost one memory round trip per 64 blocks, not one each
  constexpr int EG = kScanGroup;
  constexpr int NT = 64 * kScanWaves;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int E = a.E;
  for (int e = tid; e < E; e += NT) rank_s[e] = 0;  // first read after the next barrier
  if (a.logits != nullptr) {
    // per expert: exclusive scan of its block counts, 64 blocks at a time
    for (int e0 = wave; e0 < E; e0 += EG * kScanWaves) {
      int run[EG];
#pragma unroll
      for (int j = 0; j < EG; ++j) run[j] = 0;
      for (int B0 = 0; B0 < nblk; B0 += 64) {
        const int b = B0 + lane;
        int cv[EG];
#pragma unroll
        for (int j = 0; j < EG; ++j)  // clamped: every load in bounds, used only in range
          cv[j] = a.blk[static_cast<size_t>(min(e0 + kScanWaves * j, E - 1)) * a.nblk_cap + min(b, nblk - 1)];
#pragma unroll
        for (int j = 0; j < EG; ++j) {
          const int e = e0 + kScanWaves * j;
          const int c = b < nblk ? cv[j] : 0;
          int incl = c;
#pragma unroll
          for (int s = 1; s < 64; s <<= 1) {
            const int o = __shfl_up(incl, s, 64);
            if (lane >= s) incl += o;
          }
          if (e < E && b < nblk) a.blk[static_cast<size_t>(e) * a.nblk_cap + b] = run[j] + incl - c;
          run[j] += lane_read(incl, 63);
        }
      }
#pragma unroll
      for (int j = 0; j < EG; ++j)
        if (lane == 0 && e0 + kScanWaves * j < E) tot[e0 + kScanWaves * j] = run[j];
    }
  }
  if (a.logits_pred != nullptr) {
    // per expert: lanes sum blocks lane, lane + 64, ... in order, then a
    // fixed halving tree over the lanes
    for (int e0 = wave; e0 < E; e0 += EG * kScanWaves) {
      float sc[EG];
#pragma unroll
      for (int j = 0; j < EG; ++j) sc[j] = 0.0f;
      for (int B0 = 0; B0 < nblk; B0 += 64) {
        const int b = B0 + lane;
        float pv[EG];
#pragma unroll
        for (int j = 0; j < EG; ++j)  // clamped: every load in bounds, used only in range
          pv[j] = a.psc[static_cast<size_t>(min(e0 + kScanWaves * j, E - 1)) * a.nblk_cap + min(b, nblk - 1)];
#pragma unroll
        for (int j = 0; j < EG; ++j)
          if (b < nblk) sc[j] += pv[j];
      }
#pragma unroll
      for (int j = 0; j < EG; ++j) {
        float v = sc[j];
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) v = v + __shfl_down(v, s, 64);
        if (lane == 0 && e0 + kScanWaves * j < E) {
          score_s[e0 + kScanWaves * j] = v;
          key_s[e0 + kScanWaves * j] = rank_key(v, e0 + kScanWaves * j);
        }
      }
    }
  }
  __syncthreads();
  // offsets and the first host-visible copies (wave 0); prediction ranks
  // (the other waves when wave 0 has the offsets to do)
  const bool sel = a.logits != nullptr, pred = a.logits_pred != nullptr;
  if (wave == 0) {
    if (sel) scan_offsets(tot, nullptr, offs_s, E, lane);
    host_rows(a, sel ? offs_s : nullptr, pred ? score_s : nullptr, lane);
  }
  if (pred) rank_count(key_s, rank_s, E, sel ? tid - 64 : tid, sel ? NT - 64 : NT);
  __syncthreads();
  if (a.logits_pred != nullptr)
    for (int e = tid; e < E; e += NT) order_s[rank_s[e]] = e;
  __syncthreads();
  if (a.logits != nullptr)
    for (int e = tid; e <= E; e += NT) a.offsets[e] = offs_s[e];
  if (a.logits_pred != nullptr) {
    for (int i = tid; i < E; i += NT) {
      a.order[i] = order_s[i];
      a.score[i] = score_s[i];
    }
  }
  if (wave == 0) host_publish(a, pred ? order_s : nullptr, lane);
}

// Many tokens, step 3: slot s of token t (block t / TB) goes to grouped
// position offsets[e] + (earlier blocks' slots of e) + (its rank in block).
__global__ __launch_bounds__(256) void scatter_many_kernel(RouteArgs a, int TB) {
  const int s = blockIdx.x * 256 + threadIdx.x;
  if (s >= a.T * a.K) return;
  const int b = (s / a.K) / TB;
  const int e = min(max(a.idx[s], 0), a.E - 1);
  const int p = a.offsets[e] + a.blk[static_cast<size_t>(e) * a.nblk_cap + b] + a.lrank[s];
  a.perm[p] = s;
  a.pos[s] = p;
}

// ------------------------------------------------------------------- logits
//
// A logit is computed in the fixed fp32 order that makes the selection
// reproducible: lane l accumulates h[j] * w[j][e] with fma over
// j = l, l+64, ... ascending, then lane partials are added in a halving tree
// that pairs lane l with lane l+s for s = 32, 16, ..., 1 (lane 0 ends with
// the result); a bias is added once afterwards.
//
// Few tokens (T < kManyTokens): one wave per (router, token, expert) logit,
// lane l running residue l's fma chain from h and the transposed router
// (coalesced 128-byte rows), kWaveSteps steps of loads in flight per batch,
// then the halving tree -- the order above with no LDS staging, so a logit
// costs about one memory round trip per STEPS * 64 elements of d.
// Logit o of the launch: router o / (T E), token and expert from the rest.
constexpr int kWaveSteps = 64;

template <typename W, int STEPS>
__device__ __forceinline__ float wave_logit(const LogitsArgs& a, int o, int lane) {
  const int per = a.T * a.E;
  const int mat = o / per, te = o - mat * per;
  const int t = te / a.E, e = te - t * a.E;
  const W* hrow = static_cast<const W*>(a.h) + static_cast<size_t>(t) * a.d + lane;
  const W* wrow = static_cast<const W*>(mat == 0 ? a.wt : a.wt2) + static_cast<size_t>(e) * a.d + lane;
  const float* bias = mat == 0 ? a.bias : a.bias2;
  const int steps = a.d / 64;
  float acc = 0.0f;
  for (int s0 = 0; s0 < steps; s0 += STEPS) {
    float hv[STEPS], wv[STEPS];
#pragma unroll
    for (int u = 0; u < STEPS; ++u) {
      const int su = min(s0 + u, steps - 1);  // clamped: every load in bounds, used only in range
      hv[u] = to_f32(hrow[static_cast<size_t>(su) * 64]);
      wv[u] = to_f32(wrow[static_cast<size_t>(su) * 64]);
    }
#pragma unroll
    for (int u = 0; u < STEPS; ++u)
      if (s0 + u < steps) acc = fmaf(hv[u], wv[u], acc);
  }
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) acc = acc + __shfl_down(acc, s, 64);
  if (bias != nullptr) acc = acc + bias[e];
  return acc;  // valid in lane 0
}

template <typename W>
__global__ __launch_bounds__(256) void logits_wave_kernel(LogitsArgs a) {
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int per = a.T * a.E;
  if (o >= per * (a.wr2 != nullptr ? 2 : 1)) return;  // whole waves only: no barrier below
  const float v = wave_logit<W, kWaveSteps>(a, o, lane);
  if (lane == 0) {
    const int mat = o / per, te = o - mat * per;
    (mat == 0 ? a.logits : a.logits2)[te] = v;
  }
}

// Few tokens: a work-group takes a block of TB tokens, staged once in LDS as
// fp32, transposed (row (t, lane l) holds elements l, l + 64, ... of token
// t, few_pitch(d) bytes apart), and one (router, expert) per wave: lane l
// requests its router elements l + 64 s a batch at a time and runs the TB
// fma chains of residue l side by side, each in the order above; then the
// same halving tree per token.  So every logit has the bits of
// logits_wave_kernel, from one router load per TB tokens instead of one
// load of the router and of the token row per logit.
constexpr int kFewWaves = 4;
constexpr int kFewBatch = 64;              // router steps requested together
constexpr int kFewLdsBytes = 80 * 1024;    // staged token rows of a work-group
constexpr int kFewMinWgs = 64;             // the token block shrinks below this grid size
__host__ __device__ constexpr int few_pitch(int d) { return ((d / 64) * 4 + 15) / 16 * 16 + 16; }

template <typename W, int TB>
__global__ __launch_bounds__(64 * kFewWaves) void logits_few_kernel(LogitsArgs a) {
  constexpr int VE = 16 / static_cast<int>(sizeof(W));
  extern __shared__ __align__(16) unsigned char few_lds[];
  float* hT = reinterpret_cast<float*>(few_lds);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d, steps = d / 64, pf = few_pitch(d) / 4;
  const int t0 = blockIdx.x * TB, nt = min(TB, a.T - t0);
  // stage the block's token rows (16 bytes per thread and pass)
  const int pieces = nt * d / VE;
  for (int i = tid; i < pieces; i += 64 * kFewWaves) {
    const int j0 = i * VE, t = j0 / d, j = j0 - t * d;
    const uint4 hp = ld16(static_cast<const W*>(a.h) + static_cast<size_t>(t0) * d + j0);
    const uint32_t hw[4] = {hp.x, hp.y, hp.z, hp.w};
#pragma unroll
    for (int c = 0; c < VE; ++c) {
      const float v = sizeof(W) == 2 ? __uint_as_float((c & 1) ? (hw[c / 2] & 0xffff0000u) : (hw[c / 2] << 16))
                                     : __uint_as_float(hw[c]);
      hT[(t * 64 + (j + c) % 64) * pf + (j + c) / 64] = v;
    }
  }
  const int mats = a.wr2 != nullptr ? 2 : 1;
  const int o = blockIdx.y * kFewWaves + wave;  // (router, expert) of this wave
  const bool live = o < a.E * mats;
  const int mat = live ? o / a.E : 0, e = live ? o - mat * a.E : 0;
  const W* wrow = static_cast<const W*>(mat == 0 ? a.wt : a.wt2) + static_cast<size_t>(e) * d + lane;
  W wv[kFewBatch];
#pragma unroll
  for (int u = 0; u < kFewBatch; ++u) wv[u] = wrow[static_cast<size_t>(min(u, steps - 1)) * 64];  // clamped: in bounds
  __syncthreads();
  if (!live) return;  // whole waves, after the only barrier
  float acc[TB];
#pragma unroll
  for (int t = 0; t < TB; ++t) acc[t] = 0.0f;
  for (int s0 = 0; s0 < steps; s0 += kFewBatch) {
    if (s0 != 0) {
#pragma unroll
      for (int u = 0; u < kFewBatch; ++u)
        wv[u] = wrow[static_cast<size_t>(min(s0 + u, steps - 1)) * 64];  // clamped: in bounds, used only in range
    }
#pragma unroll
    for (int u0 = 0; u0 < kFewBatch; u0 += 4) {
      if (s0 + u0 >= steps) break;
      float hx[TB][4];
#pragma unroll
      for (int t = 0; t < TB; ++t) {
        const float4 q = *reinterpret_cast<const float4*>(hT + (t * 64 + lane) * pf + s0 + u0);
        hx[t][0] = q.x;
        hx[t][1] = q.y;
        hx[t][2] = q.z;
        hx[t][3] = q.w;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (s0 + u0 + u < steps) {
          const float w = to_f32(wv[u0 + u]);
#pragma unroll
          for (int t = 0; t < TB; ++t) acc[t] = fmaf(hx[t][u], w, acc[t]);
        }
      }
    }
  }
  const float* bias = mat == 0 ? a.bias : a.bias2;
  float* out = mat == 0 ? a.logits : a.logits2;
#pragma unroll
  for (int t = 0; t < TB; ++t) {
    float v = acc[t];
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) v = v + __shfl_down(v, s, 64);
    if (bias != nullptr) v = v + bias[e];
    if (lane == 0 && t < nt) out[static_cast<size_t>(t0 + t) * a.E + e] = v;
  }
}

// Many tokens: the same order, with each lane running the fma chains of 8
// consecutive residues (l = 8 m + k, k < 8, m = lane % 8) for a 4-token x
// 4-expert output tile (o = lane / 8 picks the tile), reading 16 bytes per
// row and step from h and from the transposed router [E][d].  A wave covers
// 8 tokens x 16 experts, a work-group 32 tokens x 16 experts of one router.
// The halving tree pairs residues l and l + 32, l + 16, l + 8 across lanes
// m ^ 4, m ^ 2, m ^ 1 -- each level a butterfly in which the two lanes keep
// opposite halves of the outputs -- and l + 4, + 2, + 1 inside the lane.
// TT x TE is a lane's output tile: 4 x 4 (a wave 8 tokens x 16 experts),
// or 2 x 2 (4 tokens x 8 experts) for launches that the larger tile would
// leave with too few waves; the last level of the halving tree of the 2 x 2
// tile adds across lanes m, m ^ 1 in both of them.
template <int TT, int TE>
struct LmTile {
  static constexpr int NO = TT * TE;           // outputs per lane
  static constexpr int TOKENS = 4 * 2 * TT;    // per work-group (4 waves)
  static constexpr int EXPERTS = 4 * TE;       // per work-group
  static_assert((TT == 4 && TE == 4) || (TT == 2 && TE == 2), "lane tiles");
};
constexpr int kLmBigBelowWgs = 512;  // 4 x 4 tiles when they give at least this many work-groups

template <typename W, int TT, int TE>
__global__ __launch_bounds__(256) void logits_many_kernel(LogitsArgs a) {
  using Tile = LmTile<TT, TE>;
  constexpr int NO = Tile::NO;
  constexpr int VPR = static_cast<int>(8 * sizeof(W)) / 16;  // 16-byte loads per row and step
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m = lane & 7, o = lane >> 3;
  const int nb = (a.E + Tile::EXPERTS - 1) / Tile::EXPERTS;
  const int mat = blockIdx.y / nb, eb = blockIdx.y - mat * nb;
  const W* wt = static_cast<const W*>(mat == 0 ? a.wt : a.wt2);
  const float* bias = mat == 0 ? a.bias : a.bias2;
  float* out = mat == 0 ? a.logits : a.logits2;
  const int tq0 = blockIdx.x * Tile::TOKENS + 2 * TT * wave + TT * (o >> 2);  // this lane's first token
  const int eq0 = eb * Tile::EXPERTS + TE * (o & 3);                          // this lane's first expert
  const W* hp[TT];
  const W* wp[TE];
#pragma unroll
  for (int i = 0; i < TT; ++i) hp[i] = static_cast<const W*>(a.h) + static_cast<size_t>(min(tq0 + i, a.T - 1)) * a.d + 8 * m;
#pragma unroll
  for (int i = 0; i < TE; ++i) wp[i] = wt + static_cast<size_t>(min(eq0 + i, a.E - 1)) * a.d + 8 * m;
  float acc[NO][8];
#pragma unroll
  for (int q = 0; q < NO; ++q)
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[q][k] = 0.0f;
  const int steps = a.d / 64;
  // the loads of P steps are in flight in P register sets, each reloaded
  // right after its step (the last steps reload the last one: in bounds,
  // never used); P = 2 for 4 x 4 tiles, whose accumulators take most of the
  // registers (measured on Qwen3-shaped prefill routing: 58 -> 54 us)
  constexpr int P = NO == 16 ? 2 : 4;
  uint4 hs[P][TT][VPR], ws[P][TE][VPR];
  auto load_step = [&](int st, uint4 (&hx)[TT][VPR], uint4 (&wx)[TE][VPR]) {
    const size_t off = static_cast<size_t>(64) * min(st, steps - 1);
#pragma unroll
    for (int v = 0; v < VPR; ++v) {
#pragma unroll
      for (int i = 0; i < TT; ++i) hx[i][v] = ld16(hp[i] + off + 8 / VPR * v);
#pragma unroll
      for (int i = 0; i < TE; ++i) wx[i][v] = ld16(wp[i] + off + 8 / VPR * v);
    }
  };
#pragma unroll
  for (int p = 0; p < P; ++p) load_step(p, hs[p], ws[p]);
  auto fma_step = [&](const uint4 (&hc)[TT][VPR], const uint4 (&wc)[TE][VPR]) {
    auto to8 = [&](const uint4 (&x)[VPR], float (&f)[8]) {
      if constexpr (VPR == 1) {
        unpack(x[0], f);
      } else {
        float lo[4], hi[4];
        unpack(x[0], lo);
        unpack(x[1], hi);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          f[k] = lo[k];
          f[4 + k] = hi[k];
        }
      }
    };
    float wf[TE][8];
#pragma unroll
    for (int i = 0; i < TE; ++i) to8(wc[i], wf[i]);
#pragma unroll
    for (int ti = 0; ti < TT; ++ti) {
      float hf[8];
      to8(hc[ti], hf);
#pragma unroll
      for (int ei = 0; ei < TE; ++ei)
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[TE * ti + ei][k] = fmaf(hf[k], wf[ei][k], acc[TE * ti + ei][k]);
    }
  };
  int st = 0;
  for (; st + P <= steps; st += P) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      fma_step(hs[p], ws[p]);
      load_step(st + p + P, hs[p], ws[p]);
    }
  }
  // steps % P last steps, their loads already in sets 0 .. steps % P - 1
#pragma unroll
  for (int p = 0; p < P - 1; ++p)
    if (st + p < steps) fma_step(hs[p], ws[p]);
  // residues l, l + 32 (lanes m, m ^ 4), then l + 16 (m ^ 2): each level a
  // butterfly in which the two lanes keep opposite halves of the outputs
  float r1[NO / 2][8];
  {
    const bool up = (m & 4) != 0;
#pragma unroll
    for (int j = 0; j < NO / 2; ++j)
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float send = up ? acc[j][k] : acc[j + NO / 2][k];
        const float keep = up ? acc[j + NO / 2][k] : acc[j][k];
        r1[j][k] = keep + __shfl_xor(send, 4, 64);
      }
  }
  float r2[NO / 4][8];
  {
    const bool up = (m & 2) != 0;
#pragma unroll
    for (int j = 0; j < NO / 4; ++j)
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float send = up ? r1[j][k] : r1[j + NO / 4][k];
        const float keep = up ? r1[j + NO / 4][k] : r1[j][k];
        r2[j][k] = keep + __shfl_xor(send, 2, 64);
      }
  }
  // l + 8 (m ^ 1): a butterfly again for 4 x 4 tiles (this lane then holds
  // outputs q = 2 m + j), both lanes the same sum for 2 x 2 ones (output q =
  // m / 2, written by the even lane)
  constexpr int NJ = NO == 16 ? 2 : 1;
  float r3[NJ][8];
  if constexpr (NO == 16) {
    const bool up = (m & 1) != 0;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float send = up ? r2[j][k] : r2[j + 2][k];
        const float keep = up ? r2[j + 2][k] : r2[j][k];
        r3[j][k] = keep + __shfl_xor(send, 1, 64);
      }
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) r3[0][k] = r2[0][k] + __shfl_xor(r2[0][k], 1, 64);
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const float* r = r3[j];
    float v = ((r[0] + r[4]) + (r[2] + r[6])) + ((r[1] + r[5]) + (r[3] + r[7]));
    const int q = NO == 16 ? 2 * m + j : m >> 1;
    const int t = tq0 + q / TE, e = eq0 + q % TE;
    if ((NO == 16 || (m & 1) == 0) && t < a.T && e < a.E) {
      if (bias != nullptr) v = v + bias[e];
      out[static_cast<size_t>(t) * a.E + e] = v;
    }
  }
}

// Logits launch, then the route launches (a kernel boundary, not a device-
// scope fence, hands data between the steps: with one L2 per XCD such
// fences write back and invalidate L2 and cost far more than a launch).
hipError_t launch_logits_route(const LogitsArgs& a, const RouteArgs& ra, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  const int mats = (a.wr != nullptr ? 1 : 0) + (a.wr2 != nullptr ? 1 : 0);
  if (mats == 0 || (a.wr != nullptr && a.wt == nullptr) || (a.wr2 != nullptr && a.wt2 == nullptr))
    return hipErrorInvalidValue;
  LogitsArgs b = a;
  if (a.wr == nullptr) {  // only the second router: move it to slot 0
    b.wr = a.wr2;
    b.wt = a.wt2;
    b.bias = a.bias2;
    b.logits = a.logits2;
    b.wr2 = nullptr;
    b.wt2 = nullptr;
  }
  const int TB = route_block_tokens(a.T, ra.K);
  const int nblk = (a.T + TB - 1) / TB;
  const bool many = (a.T >= kManyTokens || (ra.logits != nullptr && a.T * ra.K > kFewSlots)) && ra.lrank != nullptr && ra.blk != nullptr &&
                    ra.psc != nullptr && nblk <= ra.nblk_cap && TB * ra.K <= 64 * kSelWaves;
  if (!many && ra.logits != nullptr && a.T * ra.K > kFewSlots)
    return hipErrorInvalidValue;  // the one-work-group route holds T * K slots
  if (many) {
    using Big = LmTile<4, 4>;
    using Small = LmTile<2, 2>;
    const int nb = (a.E + Big::EXPERTS - 1) / Big::EXPERTS;
    const dim3 grid((a.T + Big::TOKENS - 1) / Big::TOKENS, nb * mats);
    if (static_cast<int64_t>(grid.x) * grid.y >= kLmBigBelowWgs) {
      if (a.dtype == kBF16)
        hipLaunchKernelGGL((logits_many_kernel<uint16_t, 4, 4>), grid, dim3(256), kGuardLds, s, b);
      else
        hipLaunchKernelGGL((logits_many_kernel<float, 4, 4>), grid, dim3(256), kGuardLds, s, b);
    } else {
      const int nbs = (a.E + Small::EXPERTS - 1) / Small::EXPERTS;
      const dim3 gs((a.T + Small::TOKENS - 1) / Small::TOKENS, nbs * mats);
      if (a.dtype == kBF16)
        hipLaunchKernelGGL((logits_many_kernel<uint16_t, 2, 2>), gs, dim3(256), kGuardLds, s, b);
      else
        hipLaunchKernelGGL((logits_many_kernel<float, 2, 2>), gs, dim3(256), kGuardLds, s, b);
    }
  } else {
    const int n_out = a.T * a.E * mats;
    // tokens per work-group: up to four, fewer while the grid would have
    // under kFewMinWgs work-groups (few experts: the waves would not cover
    // enough CUs)
    int tb = a.T >= 3 ? 4 : a.T;
    const int ey = (a.E * mats + kFewWaves - 1) / kFewWaves;
    while (tb > 1 && ((a.T + tb - 1) / tb) * ey < kFewMinWgs) tb /= 2;
    const size_t few_bytes = static_cast<size_t>(tb) * 64 * few_pitch(a.d);
    if (few_bytes <= kFewLdsBytes) {
      const dim3 grid((a.T + tb - 1) / tb, (a.E * mats + kFewWaves - 1) / kFewWaves);
#define MSK_FEW(TB_)                                                                                      \
  if (a.dtype == kBF16)                                                                                   \
    hipLaunchKernelGGL((logits_few_kernel<uint16_t, TB_>), grid, dim3(64 * kFewWaves), few_bytes, s, b); \
  else                                                                                                    \
    hipLaunchKernelGGL((logits_few_kernel<float, TB_>), grid, dim3(64 * kFewWaves), few_bytes, s, b)
      if (tb == 1) {
        MSK_FEW(1);
      } else if (tb == 2) {
        MSK_FEW(2);
      } else {
        MSK_FEW(4);
      }
#undef MSK_FEW
    } else {
      const dim3 grid((n_out + 3) / 4);
      if (a.dtype == kBF16)
        hipLaunchKernelGGL(logits_wave_kernel<uint16_t>, grid, dim3(256), kGuardLds, s, b);
      else
        hipLaunchKernelGGL(logits_wave_kernel<float>, grid, dim3(256), kGuardLds, s, b);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int qn = lanes_q(ra.E);
  if (!many) {
    auto* k = qn == 1 ? route_kernel<1> : qn == 2 ? route_kernel<2> : qn == 4 ? route_kernel<4> : route_kernel<8>;
    hipLaunchKernelGGL(k, dim3(1), dim3(64 * kRouteWaves), 0, s, ra);
    return hipGetLastError();
  }
  auto* sel = qn == 1   ? select_many_kernel<1>
              : qn == 2 ? select_many_kernel<2>
              : qn == 4 ? select_many_kernel<4>
                        : select_many_kernel<8>;
  if (TB > kSelWaves) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sel, dim3(nblk), dim3(64 * kSelWaves), 0, s, ra, TB);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(scan_many_kernel, dim3(1), dim3(64 * kScanWaves), 0, s, ra, nblk);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (ra.logits != nullptr) {
    hipLaunchKernelGGL(scatter_many_kernel, dim3((a.T * ra.K + 255) / 256), dim3(256), kGuardLds, s, ra, TB);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

// --------------------------------------------------------------- SwiGLU FFN
//
// A work-group computes UPW units (one sub-range of a 64-unit chunk c) of one
// expert for one tile of at most NT of the expert's tokens (the tiles of an
// expert with more tokens go to neighbouring work-groups):
//   phase 1: a[t][f] = silu(h_t . G_f) * (h_t . U_f) for its units f
//            (8 lanes per unit row, 16-byte loads, batches of RB loads per
//            lane and row stream issued before use);
//   phase 2: y[t][:] = sum_f a[t][f] * D_f over its units (each thread owns
//            VEC columns per pass);
//   writes y as the fp32 partial row of (token, plane c * subs + sub).
// Chunk layout (model dtype): [G][U][D], 64 x d elements each.  G and U are
// k-tiled: element (unit f, k) sits at ((k / 64) * 64 + f) * 64 + k % 64, so
// the units' pieces of one 64-wide k slice are adjacent; D is row-major
// (down row f at f * d).  The same code serves resident and streamed chunks,
// and a given chunk is always split the same way, so its partials do not
// depend on which launch computed it.  Loads run one batch ahead of use;
// the batch depth RB only changes how many are in flight, not the order of
// any sum: launches with several work-groups per CU use RB = 4, launches
// of fewer work-groups than CUs or of one (whole-chunk) work-group per CU
// use RB = 8 (each work-group alone must keep enough bytes in flight to
// cover the latency).

// Index of the task holding work-group wg: the last task whose first
// work-group is <= wg (tasks in ascending wg_begin order).
template <typename TaskT>
__device__ __forceinline__ int find_task_of(const TaskT* tasks, int n, int wg) {
  // the starts are ascending from 0: the task is the count of starts <= wg,
  // less one; every lane reads up to four starts at once (no chain of
  // dependent reads)
  const int lane = threadIdx.x & 63;
  int b[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) b[j] = tasks[min(64 * j + lane, n - 1)].wg_begin;  // clamped: in bounds
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) cnt += __popcll(__ballot(64 * j + lane < n && b[j] <= wg));
  return __builtin_amdgcn_readfirstlane(cnt - 1);
}

constexpr int kRowBatch = 4;        // RB of launches that fill the GPU
constexpr int kRowBatchDeep = 8;    // RB where one work-group per CU carries the loads
constexpr int kDeepBelowWgs = 256;
constexpr int kLpu = kFfnLanesPerUnit;
constexpr int kKTile = 64;                // k elements per gate/up piece

// One tile of NTT token rows (nt <= NTT real, the rest zero) of one chunk
// sub-range.  Each token's sums run in the same order whatever NTT is, so a
// token's partial does not depend on the tile it was computed in.
template <typename W, int NTT, int Q, int UPW, int RB>
__device__ __forceinline__ void ffn_tile(const FfnArgs& a, const W* G, const W* U, const W* D, float* part,
                                         int a_planes, int plane, bool routed, int p0, int tile, int nt, W* hs,
                                         float* as, int sub) {
  constexpr int VEC = Vec<W>::N;
  constexpr int THREADS = UPW * kLpu;
  constexpr int STEP = kLpu * VEC;  // k covered by the lanes of a unit per step
  constexpr int PB = (RB < 16 / Q) ? RB : 16 / Q;  // phase-2 rows per batch (<= 2 x 16 loads in flight)
  static_assert(STEP <= kKTile && kKTile % STEP == 0, "a unit's lanes must tile a k piece");
  static_assert(UPW % PB == 0, "phase-2 batches must tile the work-group's units");
  const int d = a.d;
  const W* hsrc = static_cast<const W*>(a.h);
  const int tid = threadIdx.x;
  const int lane_u = tid % kLpu;           // lane within the unit's lane group
  const int lu = tid / kLpu;               // unit within this work-group
  const int unit = sub * UPW + lu;         // unit within the chunk
  const int f_first = sub * UPW;           // first down row of this work-group
  const int n_steps = d / STEP;

  // gate/up loads of one batch of RB steps (clamped to the last step; used
  // only in range)
  auto load_batch = [&](int s0, uint4(&g)[RB], uint4(&uu)[RB]) {
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      const int sk = min(s0 + u, n_steps - 1) * STEP;  // first k of the step
      const size_t off =
          (static_cast<size_t>(sk / kKTile) * kChunkUnits + unit) * kKTile + (sk % kKTile) + lane_u * VEC;
      g[u] = ldw16(G + off);
      uu[u] = ldw16(U + off);
    }
  };
  // down-row loads of one batch of PB rows (clamped to the work-group's last)
  auto load_rows = [&](int f0, uint4(&dd)[PB][Q]) {
#pragma unroll
    for (int u = 0; u < PB; ++u)
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int col = min((tid + THREADS * q) * VEC, d - VEC);  // clamped; used only if in range
        dd[u][q] = ldw16(D + static_cast<size_t>(f_first + min(f0 + u, UPW - 1)) * d + col);
      }
  };

  // the first weight batch is requested before the activations are staged,
  // so that no work-group waits on the activation load with nothing in flight
  uint4 gn[RB], un[RB];
  load_batch(0, gn, un);

  // stage the tile's activations in LDS (zero rows past nt)
  const int vec_per_row = d / VEC;
  for (int i = tid; i < NTT * vec_per_row; i += THREADS) {
    const int t = i / vec_per_row, k = (i - t * vec_per_row) * VEC;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (t < nt) {
      const int tok = routed ? a.perm[p0 + tile + t] / a.K : tile + t;
      v = ld16(hsrc + static_cast<size_t>(tok) * d + k);
    }
    *reinterpret_cast<uint4*>(hs + static_cast<size_t>(t) * d + k) = v;
  }
  __syncthreads();

  // phase 1: gate/up dot products of this lane group's unit
  uint4 dn[PB][Q];
  {
    float ag[NTT], au[NTT];
#pragma unroll
    for (int t = 0; t < NTT; ++t) ag[t] = au[t] = 0.0f;
    // software pipeline: batch s0 + RB is loaded while batch s0 is used
    uint4 gr[RB], ur[RB];
    for (int s0 = 0; s0 < n_steps; s0 += RB) {
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        gr[u] = gn[u];
        ur[u] = un[u];
      }
      load_batch(s0 + RB, gn, un);
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        if (s0 + u < n_steps) {
          const int k = (s0 + u) * STEP + lane_u * VEC;
          float gv[VEC], uv[VEC];
          unpack(gr[u], gv);
          unpack(ur[u], uv);
#pragma unroll
          for (int t = 0; t < NTT; ++t) {
            float hv[VEC];
            unpack(ld16(hs + static_cast<size_t>(t) * d + k), hv);
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
              ag[t] = fmaf(gv[i], hv[i], ag[t]);
              au[t] = fmaf(uv[i], hv[i], au[t]);
            }
          }
        }
      }
    }
    // the first down rows are requested before the phase boundary
    load_rows(0, dn);
#pragma unroll
    for (int t = 0; t < NTT; ++t) {
#pragma unroll
      for (int s = 1; s < kLpu; s <<= 1) {
        ag[t] += __shfl_xor(ag[t], s, 64);
        au[t] += __shfl_xor(au[t], s, 64);
      }
    }
    if (lane_u == 0) {
#pragma unroll
      for (int t = 0; t < NTT; ++t) as[t * UPW + lu] = silu(ag[t]) * au[t];
    }
  }
  __syncthreads();

  // phase 2: partial down-projection over this work-group's units
  {
    float y[NTT][Q][VEC];
#pragma unroll
    for (int t = 0; t < NTT; ++t)
#pragma unroll
      for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int i = 0; i < VEC; ++i) y[t][q][i] = 0.0f;
    // software pipeline as in phase 1
    uint4 dr[PB][Q];
    for (int f0 = 0; f0 < UPW; f0 += PB) {
#pragma unroll
      for (int u = 0; u < PB; ++u)
#pragma unroll
        for (int q = 0; q < Q; ++q) dr[u][q] = dn[u][q];
      load_rows(f0 + PB, dn);
#pragma unroll
      for (int u = 0; u < PB; ++u) {
        float av[NTT];
#pragma unroll
        for (int t = 0; t < NTT; ++t) av[t] = as[t * UPW + f0 + u];
#pragma unroll
        for (int q = 0; q < Q; ++q) {
          const int col = (tid + THREADS * q) * VEC;
          if (col < d) {
            float dv[VEC];
            unpack(dr[u][q], dv);
#pragma unroll
            for (int t = 0; t < NTT; ++t)
#pragma unroll
              for (int i = 0; i < VEC; ++i) y[t][q][i] = fmaf(av[t], dv[i], y[t][q][i]);
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NTT; ++t) {
      if (t < nt) {
        const int row = routed ? (p0 + tile + t) : (tile + t);
        float* dst = part + (static_cast<size_t>(row) * a_planes + plane) * d;
#pragma unroll
        for (int q = 0; q < Q; ++q) {
          const int col = (tid + THREADS * q) * VEC;
          if (col < d) {
#pragma unroll
            for (int i = 0; i < VEC; i += 4)
              *reinterpret_cast<float4*>(dst + col + i) =
                  make_float4(y[t][q][i], y[t][q][i + 1], y[t][q][i + 2], y[t][q][i + 3]);
          }
        }
      }
    }
  }
  __syncthreads();
}

// Tiles of 5 to 16 bf16 rows run on the matrix cores in both phases
// (v_mfma_f32_16x16x32_bf16; A = the tile's rows, the last real row repeated
// past nt, whose results are never stored):
//   phase 1: B = 16 units of the chunk's k-tiled G and U rows: lane l holds
//            unit / row l % 16 and the 8 k values 8 (l / 16) + [0, 8) of a
//            32-wide k block, the A fragments loaded straight from the
//            activation rows (shared by every work-group of the expert, so
//            they come from L2).  Wave w works on unit block w % NB over every
//            other 64-wide k piece from w / NB; the sums over the even and
//            the odd pieces are added in LDS (even + odd), then the SwiGLU
//            product a[t][f] (fp32, LDS).
//   phase 2: y[t][col] = sum_f a[t][f] D[f][col], contracted over f in steps
//            of 32 units.  Lane (n, g) loads down rows 8 g .. 8 g + 7 of the
//            step at columns 8 n .. 8 n + 7 of a 128-column block (eight
//            16-byte pieces, 256 contiguous bytes per row and 16 lanes),
//            transposes them in registers into eight B fragments (column
//            8 n + j, j = 0..7) and runs one MFMA per fragment, so that its
//            results are rows 4 g .. 4 g + 3 of columns 8 n .. 8 n + 7.  a
//            enters as the bf16 pair hi + lo (hi = a rounded to bf16, lo = the
//            remainder rounded to bf16; both products are exact in fp32), so
//            16 bits of a's mantissa reach the sums.  Wave w takes the column
//            blocks w, w + waves, ...; with 16 units per work-group the step
//            is half full and its other half is zero.
// Every row's weights are read once per tile, whatever its height up to 16.
// Which path a tile takes depends only on its row count, so a token's
// partial is the same in every launch.
constexpr int kMmaTileRows = 16;
constexpr int kDnCols = 128;  // columns of one phase-2 block: 16 lanes x 8

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// fp32 -> bf16, round to nearest even (finite values)
__device__ __forceinline__ uint16_t f2bf(float f) {
  const uint32_t u = __float_as_uint(f);
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Eight rows of eight bf16 (one 16-byte piece each) -> eight column
// fragments: frag[j] = element j of rows 0 .. 7, in row order (v_perm_b32
// picks the low or high half of word j / 2 of two rows at a time).
__device__ __forceinline__ void transpose8x8(const uint4 (&rows)[8], uint4 (&frag)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
    uint32_t w[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const uint4 v = rows[r];
      w[r] = (j >> 1) == 0 ? v.x : (j >> 1) == 1 ? v.y : (j >> 1) == 2 ? v.z : v.w;
    }
    frag[j] = make_uint4(__builtin_amdgcn_perm(w[1], w[0], sel), __builtin_amdgcn_perm(w[3], w[2], sel),
                         __builtin_amdgcn_perm(w[5], w[4], sel), __builtin_amdgcn_perm(w[7], w[6], sel));
  }
}

// LDS of an FFN launch of NT-row tiles.  fma-chain tiles: activation rows
// [nt][d] and SwiGLU values [nt][upw].  Launches of kMmaTileRows bf16 rows
// run tiles of up to 4 rows on fma chains and larger ones on the matrix
// cores (SwiGLU values [16][upw] and the even/odd k exchange, 8 floats per
// lane of each unit block).
__host__ __device__ constexpr size_t ffn_lds_fma(int nt, int d, int elem, int upw) {
  return static_cast<size_t>(nt) * d * elem + sizeof(float) * nt * upw;
}
__host__ __device__ constexpr size_t ffn_lds_mma(int upw) {
  return sizeof(float) * (static_cast<size_t>(kMmaTileRows) * upw + (upw / 16) * 64 * 8);
}
__host__ __device__ constexpr size_t ffn_lds_bytes(int nt, int d, int elem, int upw) {
  return (nt == kMmaTileRows && elem == 2)
             ? (ffn_lds_fma(4, d, elem, upw) > ffn_lds_mma(upw) ? ffn_lds_fma(4, d, elem, upw) : ffn_lds_mma(upw))
             : ffn_lds_fma(nt, d, elem, upw);
}

template <int UPW>
__device__ __forceinline__ void ffn_tile_mma(const FfnArgs& a, const uint16_t* G, const uint16_t* U,
                                             const uint16_t* D, float* part, int a_planes, int plane, bool routed,
                                             int p0, int tile, int nt, float* as, float* red, int sub) {
  using W = uint16_t;
  constexpr int THREADS = UPW * kLpu;
  constexpr int NWV = THREADS / 64;  // waves
  constexpr int NB = UPW / 16;       // unit blocks, two waves each
  constexpr int KB = 2;              // k pieces per phase-1 load batch
  constexpr int S = (UPW + 31) / 32;  // 32-unit steps of phase 2
  static_assert(NWV == 2 * NB, "two waves per unit block");
  const int d = a.d;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ub = wave % NB, kh = wave / NB;
  const int n = lane & 15, g = lane >> 4;
  const int unit = sub * UPW + ub * 16 + n;
  const int f_first = sub * UPW;
  const int n_kt = d / kKTile;
  const int npw = (n_kt - kh + 1) / 2;  // k pieces of this wave: kh, kh + 2, ...
  const int ncb = (d + kDnCols - 1) / kDnCols;
  const int nblk = wave < ncb ? (ncb - 1 - wave) / NWV + 1 : 0;  // column blocks of this wave
  // lanes g >= 2 pad a half step (16 units per work-group) with zeros
  const bool k_live = UPW >= 32 || g < 2;

  // this lane's A row: tile row n, the last real row past nt
  const int ar = min(n, nt - 1);
  const int tok = routed ? a.perm[p0 + tile + ar] / a.K : tile + ar;
  const W* hrow = static_cast<const W*>(a.h) + static_cast<size_t>(tok) * d + g * 8;

  auto load_b = [&](int i0, uint4(&ba)[KB][2], uint4(&bg)[KB][2], uint4(&bu)[KB][2]) {
#pragma unroll
    for (int i = 0; i < KB; ++i) {
      // clamped (also when this wave has no piece, d = 64); used only in range
      const int kt = min(kh + 2 * max(0, min(i0 + i, npw - 1)), n_kt - 1);
      const size_t off = (static_cast<size_t>(kt) * kChunkUnits + unit) * kKTile + g * 8;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        ba[i][j] = ld16(hrow + kt * kKTile + 32 * j);
        bg[i][j] = ldw16(G + off + 32 * j);
        bu[i][j] = ldw16(U + off + 32 * j);
      }
    }
  };
  // phase-2 down rows of column block bi (of this wave) and step s
  auto load_d = [&](int bi, int s, uint4(&dd)[8]) {
    const int col = min((wave + NWV * bi) * kDnCols + 8 * n, d - 8);  // clamped; stored only if in range
    const W* src = D + static_cast<size_t>(f_first + 32 * s + 8 * g) * d + col;
#pragma unroll
    for (int r = 0; r < 8; ++r) dd[r] = k_live ? ldw16(src + static_cast<size_t>(r) * d) : make_uint4(0, 0, 0, 0);
  };

  uint4 dn[8];
  {
    f32x4_t cg = {0.0f, 0.0f, 0.0f, 0.0f}, cu = {0.0f, 0.0f, 0.0f, 0.0f};
    uint4 ban[KB][2], bgn[KB][2], bun[KB][2];
    load_b(0, ban, bgn, bun);
    for (int i0 = 0; i0 < npw; i0 += KB) {
      uint4 bar[KB][2], bgr[KB][2], bur[KB][2];
#pragma unroll
      for (int i = 0; i < KB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          bar[i][j] = ban[i][j];
          bgr[i][j] = bgn[i][j];
          bur[i][j] = bun[i][j];
        }
      load_b(i0 + KB, ban, bgn, bun);
#pragma unroll
      for (int i = 0; i < KB; ++i) {
        if (i0 + i < npw) {
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            cg = mfma16(as_bf16x8(bar[i][j]), as_bf16x8(bgr[i][j]), cg);
            cu = mfma16(as_bf16x8(bar[i][j]), as_bf16x8(bur[i][j]), cu);
          }
        }
      }
    }
    // the first down rows are requested before the k halves meet
    if (nblk > 0) load_d(0, 0, dn);
    if (kh == 1) {
      float* r = red + (static_cast<size_t>(ub) * 64 + lane) * 8;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        r[i] = cg[i];
        r[4 + i] = cu[i];
      }
    }
    __syncthreads();
    if (kh == 0) {
      const float* r = red + (static_cast<size_t>(ub) * 64 + lane) * 8;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float sg = cg[i] + r[i], su = cu[i] + r[4 + i];
        as[(4 * g + i) * UPW + ub * 16 + n] = silu(sg) * su;
      }
    }
  }
  __syncthreads();

  // phase 2: A fragments (row n, units 32 s + 8 g + [0, 8)) as hi / lo bf16
  bf16x8_t ahi[S], alo[S];
#pragma unroll
  for (int s = 0; s < S; ++s) {
    uint32_t hw[4] = {0u, 0u, 0u, 0u}, lw[4] = {0u, 0u, 0u, 0u};
    if (k_live) {
      const float* src = as + n * UPW + 32 * s + 8 * g;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float v = src[i];
        const uint16_t hb = f2bf(v);
        const float hf = bf2f(hb);
        const uint16_t lb = isfinite(hf) ? f2bf(v - hf) : static_cast<uint16_t>(0);
        hw[i >> 1] |= static_cast<uint32_t>(hb) << (16 * (i & 1));
        lw[i >> 1] |= static_cast<uint32_t>(lb) << (16 * (i & 1));
      }
    }
    ahi[s] = as_bf16x8(make_uint4(hw[0], hw[1], hw[2], hw[3]));
    alo[s] = as_bf16x8(make_uint4(lw[0], lw[1], lw[2], lw[3]));
  }
  for (int bi = 0; bi < nblk; ++bi) {
    f32x4_t acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < S; ++s) {
      uint4 dr[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) dr[r] = dn[r];
      // next: the block's next step, else the next block's first (the last
      // block reloads its own: in bounds, unused)
      if (s + 1 < S)
        load_d(bi, s + 1, dn);
      else
        load_d(min(bi + 1, nblk - 1), 0, dn);
      uint4 frag[8];
      transpose8x8(dr, frag);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        acc[j] = mfma16(ahi[s], as_bf16x8(frag[j]), acc[j]);
        acc[j] = mfma16(alo[s], as_bf16x8(frag[j]), acc[j]);
      }
    }
    const int c0 = (wave + NWV * bi) * kDnCols + 8 * n;
    if (c0 < d) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 4 * g + i;
        if (t < nt) {
          const int row = routed ? (p0 + tile + t) : (tile + t);
          float* dst = part + (static_cast<size_t>(row) * a_planes + plane) * d + c0;
          *reinterpret_cast<float4*>(dst) = make_float4(acc[0][i], acc[1][i], acc[2][i], acc[3][i]);
          *reinterpret_cast<float4*>(dst + 4) = make_float4(acc[4][i], acc[5][i], acc[6][i], acc[7][i]);
        }
      }
    }
  }
  __syncthreads();
}

// Grid: n_wg x n_tiles work-groups; block b computes token tile b % n_tiles
// of work-group slot b / n_tiles, so the tiles of an expert with many tokens
// run side by side.  The tile shape
// follows the tile's real token count (1, 2, 4 or NT rows), read on the
// device, so launches enqueued before the routing is known waste no
// arithmetic on empty rows.
template <typename W, int NT, int Q, int UPW, int RB>
__global__ __launch_bounds__(UPW * kLpu) void ffn_chunk_kernel(FfnArgs a, int n_tiles) {
  extern __shared__ __align__(16) unsigned char ffn_smem[];
  const int wg = blockIdx.x / n_tiles;
  const int tile0 = blockIdx.x - wg * n_tiles;
  const FfnTaskK tk = a.tasks[find_task_of(a.tasks, a.n_tasks, wg)];
  const int local = wg - tk.wg_begin;
  const int c = tk.chunk_lo + local / a.subs;
  const int sub = local % a.subs;
  const bool routed = tk.expert >= 0;
  int p0 = 0, n_tok = a.T;
  if (routed) {
    p0 = a.offsets[tk.expert];
    n_tok = a.offsets[tk.expert + 1] - p0;
  }

  const size_t cd = static_cast<size_t>(kChunkUnits) * a.d;
  const W* G = reinterpret_cast<const W*>(tk.base + static_cast<size_t>(c) * a.chunk_bytes);
  const W* U = G + cd;
  const W* D = U + cd;
  float* part = routed ? a.part : a.part_sh + static_cast<size_t>(-1 - tk.expert) * a.sh_plane;
  // partial layout [row][plane][d]: one slot's planes are contiguous
  const int a_planes = routed ? a.n_planes : a.n_planes_sh;
  const int plane = c * a.subs + sub;

  constexpr bool kMma = (NT == kMmaTileRows && sizeof(W) == 2);
  // fma-chain tiles of NTT rows: activation rows [NTT][d], SwiGLU values
  // after them; matrix-core tiles: SwiGLU values [16][UPW], k exchange after
  W* hs = reinterpret_cast<W*>(ffn_smem);
  auto as_of = [&](int ntt) { return reinterpret_cast<float*>(ffn_smem + sizeof(W) * ntt * a.d); };

  // one tile per work-group: the launch's n_tiles * NT rows cover every
  // task's tokens (max_tok bounds them)
  const int tile = tile0 * NT;
  if (tile >= n_tok) return;
  {
    const int nt = min(NT, n_tok - tile);
#define MSK_FFN_TILE(NTT) ffn_tile<W, NTT, Q, UPW, RB>(a, G, U, D, part, a_planes, plane, routed, p0, tile, nt, hs, as_of(NTT), sub)
    if (NT >= 4 && nt == 1) {
      MSK_FFN_TILE((NT >= 4 ? 1 : NT));
    } else if (NT >= 8 && nt <= 2) {
      MSK_FFN_TILE((NT >= 8 ? 2 : NT));
    } else if (NT >= 8 && nt <= 4) {
      MSK_FFN_TILE((NT >= 8 ? 4 : NT));
    } else if constexpr (kMma) {
      float* as = reinterpret_cast<float*>(ffn_smem);
      ffn_tile_mma<UPW>(a, reinterpret_cast<const uint16_t*>(G), reinterpret_cast<const uint16_t*>(U),
                        reinterpret_cast<const uint16_t*>(D), part, a_planes, plane, routed, p0, tile, nt, as,
                        as + kMmaTileRows * UPW, sub);
    } else {
      MSK_FFN_TILE(NT);
    }
#undef MSK_FFN_TILE
  }
}

// At most kFfnWavesPerCu waves of one FFN launch share a CU: each
// work-group streams its own weight slice once, and more concurrent streams
// per CU made the launch slower.  Measured with every expert resident, from
// the register-limited occupancy down to 8 waves per CU: DeepSeek-V2-Lite-
// shaped decode 38 -> 30 us (10 -> 4 two-wave work-groups per CU; 6 or more
// were slow), Qwen3-shaped batch 16 63 -> 62 us (2 four-wave work-groups),
// Mixtral-shaped 125 -> 123 us (one eight-wave work-group).  A launch asks
// for LDS (kLdsPerCu per CU) of 1 / (n + 1/2) of the CU for n work-groups,
// so that n fit and n + 1 do not whatever the allocation granule (up to
// 2 KiB).
constexpr int kFfnWavesPerCu = 8;
constexpr size_t kLdsPerCu = 160 * 1024;

template <typename W, int NT, int Q, int UPW>
static hipError_t launch_ffn_one(const FfnArgs& a, int max_tok, hipStream_t s) {
  size_t lds = ffn_lds_bytes(NT, a.d, static_cast<int>(sizeof(W)), UPW);
  constexpr int kWgPerCu = kFfnWavesPerCu / (UPW * kLpu / 64);
  if constexpr (kWgPerCu >= 1) lds = std::max(lds, (2 * kLdsPerCu / (2 * kWgPerCu + 1)) & ~size_t{511});
  const int n_tiles = max(1, (max_tok + NT - 1) / NT);
  const int64_t grid = static_cast<int64_t>(a.n_wg) * n_tiles;
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  // deep batches (bf16 weights) only where few tokens and columns keep the
  // accumulators small enough to leave room for the loads in flight, and
  // where one work-group alone keeps its CU's loads in flight: launches of
  // fewer work-groups than CUs, and whole-chunk work-groups (one per CU;
  // measured on the Mixtral-shaped decode FFN: 123.5 -> 121.5 us; with two
  // or more work-groups per CU deeper batches were slower)
  if constexpr (NT <= 2 && Q <= 4 && sizeof(W) == 2) {
    if (grid < kDeepBelowWgs || kWgPerCu == 1) {
      hipLaunchKernelGGL((ffn_chunk_kernel<W, NT, Q, UPW, kRowBatchDeep>), dim3(grid), dim3(UPW * kLpu), lds, s,
                         a, n_tiles);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((ffn_chunk_kernel<W, NT, Q, UPW, kRowBatch>), dim3(grid), dim3(UPW * kLpu), lds, s, a,
                     n_tiles);
  return hipGetLastError();
}

// Accumulators the kernel can hold beside its pipelined loads: those of the
// largest fma-chain tile (4 rows in a launch of matrix-core tiles, whose own
// registers do not depend on the tile height or the column passes).
constexpr bool ffn_fits(int nt, int q, int vec) {
  return (nt == kMmaTileRows && vec == 8) ? ffn_fits(4, q, vec) : nt * q * vec <= (q >= 4 ? 32 : 64);
}

// Only the (NT, Q) pairs whose accumulators fit exist.
template <typename W, int UPW>
static hipError_t dispatch_ffn(const FfnArgs& a, int nt, int q, int max_tok, hipStream_t s) {
  constexpr int V = Vec<W>::N;
  // Q_ > 1 exists only where some d <= kMaxModelDim needs it
#define MSK_FFN_CASE(NT_, Q_)                                                                     \
  if (nt == NT_ && q == Q_) {                                                                     \
    if constexpr (ffn_fits(NT_, Q_, V) && (Q_ == 1 || UPW * kLpu * V * (Q_ / 2) < kMaxModelDim))  \
      return launch_ffn_one<W, NT_, Q_, UPW>(a, max_tok, s);                                     \
  }
  MSK_FFN_CASE(1, 1) MSK_FFN_CASE(2, 1) MSK_FFN_CASE(4, 1)
  MSK_FFN_CASE(1, 2) MSK_FFN_CASE(2, 2) MSK_FFN_CASE(4, 2)
  MSK_FFN_CASE(1, 4) MSK_FFN_CASE(2, 4) MSK_FFN_CASE(4, 4)
  MSK_FFN_CASE(1, 8) MSK_FFN_CASE(2, 8) MSK_FFN_CASE(4, 8)
  if constexpr (sizeof(W) == 2) {
    MSK_FFN_CASE(kMmaTileRows, 1) MSK_FFN_CASE(kMmaTileRows, 2) MSK_FFN_CASE(kMmaTileRows, 4)
    MSK_FFN_CASE(kMmaTileRows, 8)
  } else {
    MSK_FFN_CASE(8, 1) MSK_FFN_CASE(8, 2) MSK_FFN_CASE(8, 4) MSK_FFN_CASE(8, 8)
  }
#undef MSK_FFN_CASE
  return hipErrorInvalidValue;
}

// Tokens per tile: the smallest of {1, 2, 4, 8} (fp32 weights) or {1, 2, 4,
// kMmaTileRows} (bf16) covering max_tok, limited so that the LDS stays
// within 64 KiB and the accumulators fit.  The limit depends only on the
// shape, so every launch that can hold a tile of more than 4 rows uses the
// same NT, and such a tile takes the same path in all of them.
static int pick_nt(int max_tok, int d, int elem, int q, int vec, int upw) {
  const int cap = elem == 2 ? kMmaTileRows : 8;
  auto up = [&](int nt) { return (nt == 4 && elem == 2) ? kMmaTileRows : 2 * nt; };
  auto down = [&](int nt) { return nt == kMmaTileRows ? 4 : nt / 2; };
  int nt = 1;
  while (nt < max_tok && nt < cap) nt = up(nt);
  while (nt > 1 && (ffn_lds_bytes(nt, d, elem, upw) > 65536 || !ffn_fits(nt, q, vec))) nt = down(nt);
  return nt;
}

template <typename W>
static hipError_t launch_ffn_w(const FfnArgs& a, int max_tok, hipStream_t s) {
  constexpr int vec = Vec<W>::N;
  const int upw = kChunkUnits / a.subs;
  const int threads = upw * kLpu;
  const int q = (a.d + threads * vec - 1) / (threads * vec);
  int qq = 1;
  while (qq < q) qq <<= 1;
  if (qq > 8) return hipErrorInvalidValue;
  const int nt = pick_nt(max_tok, a.d, static_cast<int>(sizeof(W)), qq, vec, upw);
  switch (a.subs) {
    case 1: return dispatch_ffn<W, 64>(a, nt, qq, max_tok, s);
    case 2: return dispatch_ffn<W, 32>(a, nt, qq, max_tok, s);
    case 4: return dispatch_ffn<W, 16>(a, nt, qq, max_tok, s);
    default: return hipErrorInvalidValue;
  }
}

// ---------------------------------------------------- SwiGLU FFN, b-bit codes
//
// One work-group per (task, chunk), all of the expert's tokens, NT at a time.
// The dot products run on v_dot2_f32_bf16: a code pair becomes the bf16 pair
// (1 + q0 / C, 1 + q1 / C), C = 2^b (the code in the top b bits of the
// mantissa of 1.0), so that over one group
//   sum_k q_k x_k = C (acc - xsum),  acc = sum_k (1 + q_k / C) x_k,
// and the group's contribution is s (C acc - (C + z) xsum) with xsum the
// group's sum of x.  x is the bf16 activation row in phase 1 and the bf16
// rounding of the SwiGLU intermediate in phase 2.
//   phase 1: lanes of a segment (LPU lanes, GPL groups each) cover the d/64
//            groups of one unit; every lane keeps its groups of the token
//            tile in registers and walks the units, B at a time, whose sums
//            a transposing butterfly over the segment completes;
//   phase 2: one down column per thread and step, the 64 intermediate values
//            of the tile in registers; writes the fp32 partial row of plane c.

constexpr uint32_t kBf16OnePair = 0x3F803F80u;

__device__ __forceinline__ float dot2bf(uint32_t a, uint32_t b, float c) {
  typedef __bf16 bf2_t __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf2_t, a), __builtin_bit_cast(bf2_t, b), c, false);
}

// Constants in registers the compiler cannot fold: (x & m) | o with m in a
// vector and o in a scalar register compiles to one v_and_or_b32, whose
// encoding takes neither a 32-bit literal nor two scalar operands, instead
// of an AND and an OR with literals.
template <uint32_t V>
__device__ __forceinline__ uint32_t sreg_const() {
  uint32_t r;
  asm("s_mov_b32 %0, %1" : "=s"(r) : "i"(V));
  return r;
}
template <uint32_t V>
__device__ __forceinline__ uint32_t vreg_const() {
  uint32_t r;
  asm("v_mov_b32 %0, %1" : "=v"(r) : "i"(V));
  return r;
}

template <int BITS>
struct PairMasks {
  static constexpr uint32_t M = ((1u << BITS) - 1u) << (7 - BITS);
  uint32_t mask, one;
  __device__ __forceinline__ PairMasks() : mask(vreg_const<M | (M << 16)>()), one(sreg_const<kBf16OnePair>()) {}
};

// Pair j of a code word as two bf16 values 1 + q / 2^BITS.
template <int BITS, int J>
__device__ __forceinline__ uint32_t code_pair(uint32_t w, const PairMasks<BITS>& pm) {
  constexpr int SH = (7 - BITS) - J * BITS;
  const uint32_t x = SH >= 0 ? (w << (SH >= 0 ? SH : 0)) : (w >> (SH < 0 ? -SH : 0));
  return (x & pm.mask) | pm.one;
}

// acc[t] = sum over one group's code words (WPG words) of pair . x[t], for
// the NT rows x[t] (32 bf16 pairs each); each pair is formed once and used
// by every row.
template <int BITS, int WPG, int NT>
__device__ __forceinline__ void group_dot(const uint32_t (&cw)[WPG], const uint32_t (*x)[32], float (&acc)[NT],
                                          const PairMasks<BITS>& pm) {
  constexpr int PPW = 16 / BITS;  // pairs per word
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = 0.0f;
#pragma unroll
  for (int m = 0; m < WPG; ++m) {
    const uint32_t w = cw[m];
#define MSK_QP(J)                                                                 \
  if constexpr (J < PPW) {                                                        \
    const uint32_t pr = code_pair<BITS, J>(w, pm);                                \
    _Pragma("unroll") for (int t = 0; t < NT; ++t) acc[t] = dot2bf(pr, x[t][m * PPW + J], acc[t]); \
  }
    MSK_QP(0) MSK_QP(1) MSK_QP(2) MSK_QP(3) MSK_QP(4) MSK_QP(5) MSK_QP(6) MSK_QP(7)
#undef MSK_QP
  }
}

__device__ __forceinline__ float fp16_lo(uint32_t m) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(m & 0xffffu)));
}
__device__ __forceinline__ float fp16_hi(uint32_t m) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(m >> 16)));
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// B unit sums per lane -> one complete unit sum per lane: log2(B) halving
// exchanges over the segment's top lane bits, then plain butterflies.  The
// lane's unit is (lane & m1 ? B/2 : 0) + (lane & m2 ? 1 : 0) (B = 4) or
// (lane & m1 ? 1 : 0) (B = 2).
template <int LPU, int B>
__device__ __forceinline__ float seg_reduce(const float (&v)[B], int li) {
  static_assert(B == 2 || B == 4, "two or four units per batch");
  static_assert(LPU >= B, "a segment needs a lane per unit of the batch");
  constexpr int m1 = LPU / 2;
  const bool h1 = (li & m1) != 0;
  float r;
  if constexpr (B == 4) {
    constexpr int m2 = LPU / 4;
    const float a0 = (h1 ? v[2] : v[0]) + __shfl_xor(h1 ? v[0] : v[2], m1, 64);
    const float a1 = (h1 ? v[3] : v[1]) + __shfl_xor(h1 ? v[1] : v[3], m1, 64);
    const bool h2 = (li & m2) != 0;
    r = (h2 ? a1 : a0) + __shfl_xor(h2 ? a0 : a1, m2, 64);
#pragma unroll
    for (int m = LPU / 8; m >= 1; m >>= 1) r += __shfl_xor(r, m, 64);
  } else {
    r = (h1 ? v[1] : v[0]) + __shfl_xor(h1 ? v[0] : v[1], m1, 64);
#pragma unroll
    for (int m = LPU / 4; m >= 1; m >>= 1) r += __shfl_xor(r, m, 64);
  }
  return r;
}

template <int BITS, int LPU, int GPL, int NT, int B>
struct QCfg {
  static constexpr int SEG = 64 / LPU;                       // segments per wave
  static constexpr int WAVES = (64 / (SEG * B)) < 4 ? (64 / (SEG * B)) : 4;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int PASSES = 64 / (WAVES * SEG * B);     // unit batches per lane
  static constexpr int WPG = 2 * BITS;                      // code words per group (64 codes)
  static constexpr int C = 1 << BITS;
  static_assert(PASSES * WAVES * SEG * B == 64, "passes must tile the chunk's units");
};

template <int BITS, int LPU, int GPL, int NT, int B>
// two waves per SIMD: at most 256 registers per lane
__global__ __launch_bounds__((QCfg<BITS, LPU, GPL, NT, B>::THREADS)) __attribute__((amdgpu_waves_per_eu(2))) void ffn_q_kernel(FfnArgs a) {
  using Q = QCfg<BITS, LPU, GPL, NT, B>;
  constexpr int WPG = Q::WPG;
  constexpr float C = static_cast<float>(Q::C);
  __shared__ __align__(16) uint16_t act[NT][kChunkUnits];  // bf16 SwiGLU intermediate of the tile
  const int d = a.d;
  const int ngr = d / 64;  // groups per gate/up row
  const int wg = blockIdx.x;
  const FfnTaskK tk = a.tasks[find_task_of(a.tasks, a.n_tasks, wg)];
  const int c = tk.chunk_lo + (wg - tk.wg_begin);
  const int p0 = a.offsets[tk.expert];
  const int n_tok = a.offsets[tk.expert + 1] - p0;
  if (n_tok <= 0) return;

  const unsigned char* chunk = tk.base + static_cast<size_t>(c) * a.chunk_bytes;
  const size_t qrow = static_cast<size_t>(d) * BITS / 8;  // code bytes of one gate/up row
  const uint4* Gq = reinterpret_cast<const uint4*>(chunk);
  const uint4* Uq = reinterpret_cast<const uint4*>(chunk + 64 * qrow);
  const uint4* Dq = reinterpret_cast<const uint4*>(chunk + 128 * qrow);
  const uint32_t* Gm = reinterpret_cast<const uint32_t*>(chunk + 192 * qrow);
  const uint32_t* Um = Gm + 64 * ngr;
  const uint32_t* Dm = Gm + 128 * ngr;
  const uint32_t* hsrc = static_cast<const uint32_t*>(a.h);  // bf16 pairs

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int sg = lane / LPU, li = lane % LPU;
  constexpr int V4 = WPG / 4;  // uint4 loads per group
  const PairMasks<BITS> pm;

  // phase 2 reads its down columns PB at a time, one batch ahead; the first
  // batch is requested before phase 1 so that it lands meanwhile
  constexpr int PB = 4;
  const int ncol = d / Q::THREADS;
  uint4 dn[PB][V4];
  uint32_t dmn[PB];
  auto load_cols = [&](int k0) {
#pragma unroll
    for (int b = 0; b < PB; ++b) {
      const int col = tid + Q::THREADS * min(k0 + b, ncol - 1);  // clamped past the last column
#pragma unroll
      for (int v = 0; v < V4; ++v) dn[b][v] = ldw16(Dq + static_cast<size_t>(col) * V4 + v);
      dmn[b] = Dm[col];
    }
  };

  for (int tile = 0; tile < n_tok; tile += NT) {
    const int nt = min(NT, n_tok - tile);
    load_cols(0);
    // ---- phase 1
    {
      uint32_t xh[GPL][NT][32];
      float xs[GPL][NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int tok = a.perm[p0 + tile + min(t, nt - 1)] / a.K;  // clamped: rows past nt are not stored
#pragma unroll
        for (int i = 0; i < GPL; ++i) {
          const uint4* hp = reinterpret_cast<const uint4*>(hsrc + (static_cast<size_t>(tok) * d + (li + LPU * i) * 64) / 2);
#pragma unroll
          for (int v = 0; v < 8; ++v) {
            const uint4 q = hp[v];
            xh[i][t][4 * v] = q.x;
            xh[i][t][4 * v + 1] = q.y;
            xh[i][t][4 * v + 2] = q.z;
            xh[i][t][4 * v + 3] = q.w;
          }
          float sum = 0.0f;
#pragma unroll
          for (int p = 0; p < 32; ++p) sum = dot2bf(xh[i][t][p], kBf16OnePair, sum);
          xs[i][t] = sum;
        }
      }
      // code words and metadata of a batch of B units, loaded one batch ahead
      uint4 gcur[B][GPL][V4], ucur[B][GPL][V4], gnx[B][GPL][V4], unx[B][GPL][V4];
      uint32_t gmc[B][GPL], umc[B][GPL], gmn[B][GPL], umn[B][GPL];
      auto load_batch = [&](int pass, uint4(&g)[B][GPL][V4], uint4(&u)[B][GPL][V4], uint32_t(&gm)[B][GPL],
                            uint32_t(&um)[B][GPL]) {
        const int pc = min(pass, Q::PASSES - 1);  // clamped: the batch past the last is loaded, not used
        const int ub = ((pc * Q::WAVES + wave) * Q::SEG + sg) * B;
#pragma unroll
        for (int j = 0; j < B; ++j)
#pragma unroll
          for (int i = 0; i < GPL; ++i) {
            const size_t grp = static_cast<size_t>(ub + j) * ngr + li + LPU * i;
#pragma unroll
            for (int v = 0; v < V4; ++v) {
              g[j][i][v] = ldw16(Gq + grp * V4 + v);
              u[j][i][v] = ldw16(Uq + grp * V4 + v);
            }
            gm[j][i] = Gm[grp];
            um[j][i] = Um[grp];
          }
      };
      load_batch(0, gnx, unx, gmn, umn);
      for (int pass = 0; pass < Q::PASSES; ++pass) {
#pragma unroll
        for (int j = 0; j < B; ++j)
#pragma unroll
          for (int i = 0; i < GPL; ++i) {
#pragma unroll
            for (int v = 0; v < V4; ++v) {
              gcur[j][i][v] = gnx[j][i][v];
              ucur[j][i][v] = unx[j][i][v];
            }
            gmc[j][i] = gmn[j][i];
            umc[j][i] = umn[j][i];
          }
        load_batch(pass + 1, gnx, unx, gmn, umn);
        const int ub = ((pass * Q::WAVES + wave) * Q::SEG + sg) * B;
        float gv[NT][B], uv[NT][B];
#pragma unroll
        for (int j = 0; j < B; ++j) {
#pragma unroll
          for (int t = 0; t < NT; ++t) gv[t][j] = uv[t][j] = 0.0f;
#pragma unroll
          for (int i = 0; i < GPL; ++i) {
            uint32_t gw[WPG], uw[WPG];
#pragma unroll
            for (int v = 0; v < V4; ++v) {
              gw[4 * v] = gcur[j][i][v].x;
              gw[4 * v + 1] = gcur[j][i][v].y;
              gw[4 * v + 2] = gcur[j][i][v].z;
              gw[4 * v + 3] = gcur[j][i][v].w;
              uw[4 * v] = ucur[j][i][v].x;
              uw[4 * v + 1] = ucur[j][i][v].y;
              uw[4 * v + 2] = ucur[j][i][v].z;
              uw[4 * v + 3] = ucur[j][i][v].w;
            }
            float ga[NT], ua[NT];
            group_dot<BITS, WPG, NT>(gw, xh[i], ga, pm);
            group_dot<BITS, WPG, NT>(uw, xh[i], ua, pm);
            const float gs = fp16_lo(gmc[j][i]), gz = C + fp16_hi(gmc[j][i]);
            const float us = fp16_lo(umc[j][i]), uz = C + fp16_hi(umc[j][i]);
#pragma unroll
            for (int t = 0; t < NT; ++t) {
              gv[t][j] += gs * (C * ga[t] - gz * xs[i][t]);
              uv[t][j] += us * (C * ua[t] - uz * xs[i][t]);
            }
          }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const float g = seg_reduce<LPU, B>(gv[t], li);
          const float u = seg_reduce<LPU, B>(uv[t], li);
          constexpr int WR = LPU / B;  // lanes holding the same unit after the reduction
          if ((li % WR) == 0) {
            const int j = li / WR;
            act[t][ub + j] = f32_to_bf16_rne(silu(g) * u);
          }
        }
      }
    }
    __syncthreads();
    // ---- phase 2
    {
      uint32_t xa[NT][32];
      float as[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const uint4* ap = reinterpret_cast<const uint4*>(&act[t][0]);
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const uint4 q = ap[v];
          xa[t][4 * v] = q.x;
          xa[t][4 * v + 1] = q.y;
          xa[t][4 * v + 2] = q.z;
          xa[t][4 * v + 3] = q.w;
        }
        float sum = 0.0f;
#pragma unroll
        for (int p = 0; p < 32; ++p) sum = dot2bf(xa[t][p], kBf16OnePair, sum);
        as[t] = sum;
      }
      uint4 dc[PB][V4];
      uint32_t dmc[PB];
      for (int k0 = 0; k0 < ncol; k0 += PB) {
#pragma unroll
        for (int b = 0; b < PB; ++b) {
#pragma unroll
          for (int v = 0; v < V4; ++v) dc[b][v] = dn[b][v];
          dmc[b] = dmn[b];
        }
        load_cols(k0 + PB);
#pragma unroll
        for (int b = 0; b < PB; ++b) {
          if (k0 + b < ncol) {
            const int col = tid + Q::THREADS * (k0 + b);
            uint32_t dw[WPG];
#pragma unroll
            for (int v = 0; v < V4; ++v) {
              dw[4 * v] = dc[b][v].x;
              dw[4 * v + 1] = dc[b][v].y;
              dw[4 * v + 2] = dc[b][v].z;
              dw[4 * v + 3] = dc[b][v].w;
            }
            const float sc = fp16_lo(dmc[b]), zc = C + fp16_hi(dmc[b]);
            float acc[NT];
            group_dot<BITS, WPG, NT>(dw, xa, acc, pm);
#pragma unroll
            for (int t = 0; t < NT; ++t) {
              if (t < nt) {
                const int row = p0 + tile + t;
                a.part[(static_cast<size_t>(row) * a.n_planes + c) * d + col] = sc * (C * acc[t] - zc * as[t]);
              }
            }
          }
        }
      }
    }
    __syncthreads();
  }
}

// One token per tile: the pairs of a second token's dot products would
// need more registers than the work-group keeps (decode tiles hold one or
// two tokens per expert; more tokens loop over the tile).
template <int BITS, int LPU, int GPL, int B>
static hipError_t launch_ffn_q_one(const FfnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((ffn_q_kernel<BITS, LPU, GPL, 1, B>), dim3(a.n_wg), dim3(QCfg<BITS, LPU, GPL, 1, B>::THREADS), 0,
                     s, a);
  return hipGetLastError();
}

template <int BITS>
static hipError_t launch_ffn_q_bits(const FfnArgs& a, hipStream_t s) {
  constexpr int B = BITS == 2 ? 4 : 2;  // units per lane and batch: code registers in flight
  switch (a.d / 64) {
    case 4: return launch_ffn_q_one<BITS, 4, 1, B>(a, s);
    case 8: return launch_ffn_q_one<BITS, 8, 1, B>(a, s);
    case 16: return launch_ffn_q_one<BITS, 16, 1, B>(a, s);
    case 32: return launch_ffn_q_one<BITS, 32, 1, B>(a, s);
    case 64: return launch_ffn_q_one<BITS, 64, 1, B>(a, s);
    case 128: return launch_ffn_q_one<BITS, 64, 2, B>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_ffn(const FfnArgs& a, int max_tok, hipStream_t s) {
  if (a.n_wg <= 0 || a.n_tasks <= 0) return hipSuccess;
  if (a.bits != 0) {
    if (a.dtype != kBF16 || a.subs != 1 || !q_supported(a.d)) return hipErrorInvalidValue;
    for (int i = 0; i < a.n_tasks; ++i)
      if (a.tasks[i].expert < 0) return hipErrorInvalidValue;  // shared experts stay in the model dtype
    if (a.bits == 2) return launch_ffn_q_bits<2>(a, s);
    if (a.bits == 4) return launch_ffn_q_bits<4>(a, s);
    return hipErrorInvalidValue;
  }
  return (a.dtype == kBF16) ? launch_ffn_w<uint16_t>(a, max_tok, s) : launch_ffn_w<float>(a, max_tok, s);
}

// ------------------------------------------------------------ prefill MFMA
//
// (operand layout of v_mfma_f32_16x16x32_bf16: see mfma16)

// Work-groups are dispatched to the 8 XCDs round-robin by index, and each
// XCD has its own L2.  The matrix-core kernels renumber them so that every
// XCD runs a contiguous range of logical indices: consecutive indices (the
// row tiles of one chunk in gate/up, the column blocks of one row tile in
// down, and in both the work of one expert) then share an L2.  Measured on
// the Qwen3-shaped prefill: gate/up L2 hits 38% -> 64%, bytes fetched past
// L2 2.0 -> 1.1 GB per launch (the launch time did not change: these
// kernels are not bound by those fetches).
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_local(int wg, int n) {
  const int q = n / kXcds, r = n % kXcds;
  const int x = wg % kXcds, i = wg / kXcds;
  return x < r ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

__device__ __forceinline__ int find_task(const MmaTask* tasks, int n, int wg) {
  return find_task_of(tasks, n, wg);
}

// Rows of a task's row tile: routed experts take grouped positions
// [offsets[e] + 64 mt, ...), shared experts take tokens [64 mt, ...).
struct TileRows {
  int p0, n;
};
__device__ __forceinline__ TileRows tile_rows(const MmaArgs& a, const MmaTask& tk, int mt) {
  TileRows r;
  const int rows = a.tile_rows;
  if (tk.expert >= 0) {
    const int b = a.offsets[tk.expert], e = a.offsets[tk.expert + 1];
    r.p0 = b + mt * rows;
    r.n = min(rows, e - r.p0);
  } else {
    r.p0 = mt * rows;
    r.n = min(rows, a.T - r.p0);
  }
  return r;
}

// gate/up: a work-group takes 64 rows x 16 NF units (kChunkUnits / (16 NF)
// = a.gu_split work-groups per chunk and row tile); wave w the rows 16 w ..
// 16 w + 15.  Per 32-wide k step a lane loads one A fragment and NF G and NF
// U fragments; loads run one batch ahead of the MFMAs.  Launches with few
// row-tile chunks split each chunk four ways (NF = 1) for parallelism;
// large ones keep whole chunks (NF = 4), so the activation rows are read
// once per chunk.  Each activation is written once, so the split changes no
// result.
template <int NF>
__global__ __launch_bounds__(256) void mma_gateup_kernel(MmaArgs a) {
  constexpr int KB = NF == 1 ? 4 : 2;  // k steps per batch
  const int wg = xcd_local(blockIdx.x, gridDim.x);
  const MmaTask tk = a.tasks[find_task(a.tasks, a.n_tasks, wg)];
  const int local = wg - tk.wg_begin;
  const int mt = local % tk.m_tiles;
  const int cq = local / tk.m_tiles;          // chunk * split + part
  const int split = kChunkUnits / (16 * NF);
  const int c = tk.chunk_lo + cq / split, part = cq % split;
  const TileRows tr = tile_rows(a, tk, mt);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (16 * wave >= tr.n) return;  // no rows for this wave (no barrier in this kernel)
  const int d = a.d;
  const bool routed = tk.expert >= 0;
  // this lane's A row: tile row 16 wave + lane % 16 (clamped; masked at the end)
  const int ar = min(16 * wave + (lane & 15), tr.n - 1);
  const int tok = routed ? a.perm[tr.p0 + ar] / a.K : tr.p0 + ar;
  const uint16_t* hrow = static_cast<const uint16_t*>(a.h) + static_cast<size_t>(tok) * d;
  const uint16_t* G = reinterpret_cast<const uint16_t*>(tk.base + static_cast<size_t>(c) * a.chunk_bytes);
  const uint16_t* U = G + static_cast<size_t>(kChunkUnits) * d;
  const int unit0 = 16 * NF * part + (lane & 15);  // this lane's first B column (unit within the chunk)
  const int kq = 8 * (lane >> 4);                // this lane's k offset inside a 32-wide step
  f32x4_t ag[NF], au[NF];
#pragma unroll
  for (int n = 0; n < NF; ++n) ag[n] = au[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  uint4 an[KB], gn[KB][NF], un[KB][NF];
  auto load = [&](int k0) {  // steps past d reload the last one (in bounds, not used)
#pragma unroll
    for (int s = 0; s < KB; ++s) {
      const int k = min(k0 + 32 * s, d - 32);
      an[s] = ld16(hrow + k + kq);
#pragma unroll
      for (int n = 0; n < NF; ++n) {
        const size_t off =
            (static_cast<size_t>(k / kKTile) * kChunkUnits + unit0 + 16 * n) * kKTile + (k % kKTile) + kq;
        gn[s][n] = ldw16(G + off);
        un[s][n] = ldw16(U + off);
      }
    }
  };
  load(0);
  for (int k0 = 0; k0 < d; k0 += 32 * KB) {
    uint4 ac[KB], gc[KB][NF], uc[KB][NF];
#pragma unroll
    for (int s = 0; s < KB; ++s) {
      ac[s] = an[s];
#pragma unroll
      for (int n = 0; n < NF; ++n) {
        gc[s][n] = gn[s][n];
        uc[s][n] = un[s][n];
      }
    }
    load(k0 + 32 * KB);
#pragma unroll
    for (int s = 0; s < KB; ++s) {
      if (k0 + 32 * s < d) {
        const bf16x8_t A = as_bf16x8(ac[s]);
#pragma unroll
        for (int n = 0; n < NF; ++n) {
          ag[n] = mfma16(A, as_bf16x8(gc[s][n]), ag[n]);
          au[n] = mfma16(A, as_bf16x8(uc[s][n]), au[n]);
        }
      }
    }
  }
  // epilogue: act = silu(g) * u as bf16, rows 16 wave + 4 (lane / 16) + r
  uint16_t* act = routed ? a.act : a.act_sh + static_cast<size_t>(-1 - tk.expert) * a.rows_shared * a.f_pad_sh;
  const int f_pad = routed ? a.f_pad : a.f_pad_sh;
#pragma unroll
  for (int n = 0; n < NF; ++n) {
    const int f = c * kChunkUnits + unit0 + 16 * n;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 16 * wave + 4 * (lane >> 4) + r;
      if (row < tr.n) act[static_cast<size_t>(tr.p0 + row) * f_pad + f] = f2bf(silu(ag[n][r]) * au[n][r]);
    }
  }
}

// activation rows of the b-bit gate/up kernel are staged in LDS in slabs of
// kGuSlab k, rows padded so that the 16 rows a fragment read touches fall in
// distinct banks
constexpr int kGuSlab = 128;            // k per staged slab (4 MFMA k-steps)
constexpr int kGuPitch = kGuSlab + 8;   // bf16 per staged row

// gate/up with both operands staged by direct global -> LDS loads
// (global_load_lds_dwordx4: a lane's 16 bytes land at the LDS address in M0
// + 16 lane, with no register in between, so the registers hold only the
// accumulators and the fragments of one k step).  A work-group takes a pair
// or four chunks (gd_group_chunks; 64 units of G and of U each, so that every
// staged activation row feeds all of them) for a row tile of up to kGdMaxRows rows and
// takes the height of its tile: 64, 128 or 192 rows, so that an expert's
// rows usually fit one tile and its weights are read once.  The k loop runs
// over stages of 64 k in a ring of as many LDS buffers as kGdLds holds for
// that height (4, 3 or 2): the loads of all but one are in flight while a
// stage is computed.  A wave
// waits for its own loads of a stage, then a barrier makes every wave's
// loads visible and frees the buffer read before for the next loads.  The
// loads are issued from inline assembly, so the compiler, which would
// otherwise wait for every load in flight into an LDS array before reading
// any part of it, leaves the waits to the kernel.  A load moves 8 rows of
// 128 bytes (whole cache lines).  Staged rows hold 8 pieces of 8 k; piece p
// of row r sits in slot p ^ (r % 8), so the 8 lanes an LDS read serves
// together (8 rows at one piece) hit distinct banks.  The waves split the
// tile kGdWaves / 2 x 2: wave (wr, wc) takes the row blocks wr, wr +
// kGdWaves / 2, ... and all 64 units of G and of U of the chunks of half wc
// of the group (a group that runs past the task's last chunk loads that one
// again and stores nothing for it).  The k order of every sum is that of the
// other gate/up kernels.
constexpr int kGdWaves = 8;                                  // waves per work-group
constexpr int kGdLds = 160 * 1024;                           // LDS of a work-group (one per CU)
constexpr int kGdSlab = 64;                                  // k per stage
constexpr int kGdMaxRB = 12;                                 // row blocks of 16 per tile at most
constexpr int kGdRowBytes = 2 * kGdSlab;                     // one staged row: a cache line
constexpr int kGdLoadBytes = 64 * 16;                        // one load: 8 rows
constexpr int kGdBlockBytes = 16 * kGdRowBytes;              // one 16-row block
constexpr int kGdBBytes = kChunkUnits * kGdRowBytes;         // G (or U) units of a stage
static_assert(kGdMaxRB * 16 == kGdMaxRows, "tile height of the staged gate/up kernel");
static_assert(kGdSlab == kKTile, "a stage is one k piece of the gate/up layout");

// 16 bytes per lane from global memory to LDS byte address lds + 16 lane
// (lds uniform over the wave); M0 is restored for the compiler
__device__ __forceinline__ void lds_load16(const void* g, uint32_t lds) {
  uint32_t keep;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(keep)
      : "v"(g), "s"(lds)
      : "memory");
}

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)(p)));
}

// wait until at most N of this wave's vector memory loads are in flight
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// barrier without a memory fence (a fence would wait for every load in
// flight into LDS): this wave's LDS reads are complete first, and the
// clobber keeps the compiler from moving LDS accesses across it
__device__ __forceinline__ void bare_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ bf16x8_t lds_frag(const unsigned char* p) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(p));
}

template <int RB, int NC>
__device__ __forceinline__ void gd_tile(const MmaArgs& a, const MmaTask& tk, int c, int nv, const TileRows& tr,
                                        unsigned char* lds) {
  constexpr int WR = kGdWaves / 2;            // row groups of waves
  constexpr int CPW = NC / 2;                 // chunks per wave (its column group's)
  constexpr int NA = 2 * RB / kGdWaves;       // activation loads per wave and stage
  constexpr int NL = NA + 2 * NC;             // loads per wave and stage (one of each of G, U of every chunk)
  constexpr int HB = RB / WR;                 // row blocks per wave
  constexpr int ABYTES = RB * kGdBlockBytes;  // activation rows of a stage
  constexpr int SBYTES = ABYTES + 2 * NC * kGdBBytes;
  constexpr int NST = kGdLds / SBYTES;        // stages in the ring
  static_assert(kGdWaves == 8 && (NC == 2 || NC == 4), "one G and one U load of each chunk per wave and stage");
  static_assert(RB % WR == 0 && (2 * RB) % kGdWaves == 0 && RB <= kGdMaxRB, "row blocks");
  static_assert(NST >= 2 && (NST - 2) * NL < 64, "ring depth");
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = w >> 1, wc = w & 1;  // wc: the column group (chunks wc CPW ..)
  const int d = a.d, nsl = d / kGdSlab;
  const bool routed = tk.expert >= 0;
  const int lrow = lane >> 3;
  const int lpiece = (lane & 7) ^ lrow;
  const uint16_t* hsrc[NA];
#pragma unroll
  for (int j = 0; j < NA; ++j) {
    const int r = min(8 * (w + kGdWaves * j) + lrow, tr.n - 1);  // rows past the tile repeat its last (never stored)
    const int tok = routed ? a.perm[tr.p0 + r] / a.K : tr.p0 + r;
    hsrc[j] = static_cast<const uint16_t*>(a.h) + static_cast<size_t>(tok) * d + 8 * lpiece;
  }
  // chunks of the group past the task's last load that one again (never stored)
  const uint16_t* Gc[NC];
#pragma unroll
  for (int j = 0; j < NC; ++j)
    Gc[j] = reinterpret_cast<const uint16_t*>(tk.base + static_cast<size_t>(c + min(j, nv - 1)) * a.chunk_bytes) +
            (8 * w + lrow) * kKTile + 8 * lpiece;
  const size_t uo = static_cast<size_t>(kChunkUnits) * d;  // U after G
  const uint32_t lbase = lds_address(lds) + w * kGdLoadBytes;
  auto issue = [&](int sl, int buf) {  // stages past the last reload it (in bounds, never read)
    const int k0 = min(sl, nsl - 1) * kGdSlab;
    const uint32_t st = lbase + buf * SBYTES;
#pragma unroll
    for (int j = 0; j < NA; ++j) lds_load16(hsrc[j] + k0, st + kGdWaves * j * kGdLoadBytes);
    const size_t bo = static_cast<size_t>(k0) * kChunkUnits;
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      lds_load16(Gc[j] + bo, st + ABYTES + 2 * j * kGdBBytes);
      lds_load16(Gc[j] + uo + bo, st + ABYTES + (2 * j + 1) * kGdBBytes);
    }
  };
  int fo[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) fo[s] = (lane & 15) * kGdRowBytes + 16 * ((4 * s + (lane >> 4)) ^ (lane & 7));
  f32x4_t ag[HB][CPW][4], au[HB][CPW][4];
#pragma unroll
  for (int i = 0; i < HB; ++i)
#pragma unroll
    for (int q = 0; q < CPW; ++q)
#pragma unroll
      for (int n = 0; n < 4; ++n) ag[i][q][n] = au[i][q][n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) {
    const unsigned char* st = lds + buf * SBYTES;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const unsigned char* sa = st + wr * kGdBlockBytes + fo[s];
      bf16x8_t g[CPW][4], u[CPW][4];
#pragma unroll
      for (int q = 0; q < CPW; ++q) {
        const unsigned char* sg = st + ABYTES + 2 * (wc * CPW + q) * kGdBBytes + fo[s];
        const unsigned char* su = sg + kGdBBytes;
#pragma unroll
        for (int n = 0; n < 4; ++n) {
          g[q][n] = lds_frag(sg + n * kGdBlockBytes);
          u[q][n] = lds_frag(su + n * kGdBlockBytes);
        }
      }
#pragma unroll
      for (int i = 0; i < HB; ++i) {
        const bf16x8_t A = lds_frag(sa + WR * i * kGdBlockBytes);
#pragma unroll
        for (int q = 0; q < CPW; ++q)
#pragma unroll
          for (int n = 0; n < 4; ++n) {
            ag[i][q][n] = mfma16(A, g[q][n], ag[i][q][n]);
            au[i][q][n] = mfma16(A, u[q][n], au[i][q][n]);
          }
      }
    }
  };
#pragma unroll
  for (int p = 0; p < NST - 1; ++p) issue(p, p);
  int cur = 0, nxt = NST - 1;
  for (int sl = 0; sl < nsl; ++sl) {
    wait_vm<(NST - 2) * NL>();
    bare_barrier();
    issue(sl + NST - 1, nxt);
    compute(cur);
    cur = cur + 1 == NST ? 0 : cur + 1;
    nxt = nxt + 1 == NST ? 0 : nxt + 1;
  }
  wait_vm<0>();  // the reloads past the last stage land before the work-group ends
  uint16_t* act = routed ? a.act : a.act_sh + static_cast<size_t>(-1 - tk.expert) * a.rows_shared * a.f_pad_sh;
  const int f_pad = routed ? a.f_pad : a.f_pad_sh;
#pragma unroll
  for (int q = 0; q < CPW; ++q) {
    const int j = wc * CPW + q;
    if (j >= nv) continue;
#pragma unroll
    for (int i = 0; i < HB; ++i) {
      const int rb = WR * i + wr;
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const int f = (c + j) * kChunkUnits + 16 * n + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 16 * rb + 4 * (lane >> 4) + r;
          if (row < tr.n) act[static_cast<size_t>(tr.p0 + row) * f_pad + f] = f2bf(silu(ag[i][q][n][r]) * au[i][q][n][r]);
        }
      }
    }
  }
}

// this work-group's task and its index within the task, from the kernel
// arguments or from tasks planned on the device; false past the planned ones
__device__ __forceinline__ bool staged_task(const MmaArgs& a, MmaTask& tk, int& local) {
  int wg;
  if (a.dtasks) {
    const int n_wg = a.dcount[1];
    if (static_cast<int>(blockIdx.x) >= n_wg) return false;
    wg = xcd_local(blockIdx.x, n_wg);
    tk = a.dtasks[find_task(a.dtasks, a.dcount[0], wg)];
  } else {
    wg = xcd_local(blockIdx.x, gridDim.x);
    tk = a.tasks[find_task(a.tasks, a.n_tasks, wg)];
  }
  local = wg - tk.wg_begin;
  return true;
}

__global__ __launch_bounds__(64 * kGdWaves) void mma_gateup_dma_kernel(MmaArgs a) {
  __shared__ __align__(16) unsigned char lds[kGdLds];
  MmaTask tk;
  int local;
  if (!staged_task(a, tk, local)) return;
  const int mt = local % tk.m_tiles;
  const int per =
      gd_group_chunks(tk.expert >= 0 ? a.offsets[tk.expert + 1] - a.offsets[tk.expert] : a.T, tk.n_chunks);
  const int c = tk.chunk_lo + per * (local / tk.m_tiles);  // the group's first chunk
  const int nv = min(per, tk.chunk_lo + tk.n_chunks - c);   // its chunks in the task
  const TileRows tr = tile_rows(a, tk, mt);
  if (tr.n <= 0) return;  // uniform over the work-group
  if (per == 4)
    gd_tile<4, 4>(a, tk, c, nv, tr, lds);  // (a task of at most 64 rows: one tile of at most 64)
  else if (tr.n <= 64)
    gd_tile<4, 2>(a, tk, c, nv, tr, lds);
  else if (tr.n <= 128)
    gd_tile<8, 2>(a, tk, c, nv, tr, lds);
  else
    gd_tile<12, 2>(a, tk, c, nv, tr, lds);
}

// Work-group barrier that orders LDS only: a __syncthreads() also orders
// global memory, and the compiler then waits for every global load in
// flight (the next chunk's, issued just before) at the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// down: a work-group takes 64 rows x kMmaCols (256) columns over all of the
// expert's chunks; wave w the rows 16 w .. 16 w + 15.  Per chunk the
// 64 x 256 down tile is staged transposed in LDS (dt[column][unit]): thread
// (unit group u = tid % 8, column group g = tid / 8) loads units 8 u .. 8 u
// + 7 of columns 8 g .. 8 g + 7 (eight 16-byte row pieces), transposes them
// in registers (v_perm_b32) into eight 16-byte column fragments and writes
// each with one LDS store.  With a row pitch of 72 units, the 16 lanes of a
// store pass (8 unit groups x 2 column groups 8 apart) and the 16 lanes of a
// fragment read (16 consecutive columns) each hit 16 distinct bank quads.
// Two chunks' tiles are in flight ahead of the one computing: the loop has
// no branch (waves past the tile's rows compute on its last row and store
// nothing; an odd last chunk runs after the loop), barriers order LDS only,
// and no register set is copied while its loads are in flight, so the
// compiler's waits cover only the chunk being used (measured: DeepSeek-V2-
// Lite prefill 512 down 109 -> 104 us).
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void mma_down_kernel(MmaArgs a) {
  constexpr int PITCH = kChunkUnits + 8;  // transposed D tile row: 64 units + pad
  __shared__ __align__(16) uint16_t dt[kMmaCols * PITCH];
  const int wg = xcd_local(blockIdx.x, gridDim.x);
  const MmaTask tk = a.tasks[find_task(a.tasks, a.n_tasks, wg)];
  const int local = wg - tk.wg_begin;
  const int mt = local / a.ncb, cb = local % a.ncb;
  const TileRows tr = tile_rows(a, tk, mt);
  if (tr.n <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d;
  const bool routed = tk.expert >= 0;
  const uint16_t* act = routed ? a.act : a.act_sh + static_cast<size_t>(-1 - tk.expert) * a.rows_shared * a.f_pad_sh;
  const int f_pad = routed ? a.f_pad : a.f_pad_sh;
  const int ar = min(16 * wave + (lane & 15), tr.n - 1);
  const uint16_t* arow = act + static_cast<size_t>(tr.p0 + ar) * f_pad;
  const int kq = 8 * (lane >> 4);
  const int col0 = cb * kMmaCols;
  const int ug = tid & 7, cg = tid >> 3;
  const int lcol = min(col0 + 8 * cg, d - 8);  // this thread's loaded columns (clamped; never stored past d)
  constexpr int NF = kMmaCols / 16;
  f32x4_t acc[NF];
#pragma unroll
  for (int nf = 0; nf < NF; ++nf) acc[nf] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  uint4 d0[8], a0[2], d1[8], a1[2];
  auto load_d = [&](int c, uint4(&dn)[8]) {
    const unsigned char* cbase = (c < tk.split ? tk.base : tk.base2) + static_cast<size_t>(c) * a.chunk_bytes;
    const uint16_t* D = reinterpret_cast<const uint16_t*>(cbase) + 2 * static_cast<size_t>(kChunkUnits) * d;
#pragma unroll
    for (int r = 0; r < 8; ++r) dn[r] = ld16(D + static_cast<size_t>(8 * ug + r) * d + lcol);
  };
  auto load_a = [&](int c, uint4(&an)[2]) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) an[ks] = ld16(arow + c * kChunkUnits + 32 * ks + kq);
  };
  auto load_chunk = [&](int c, uint4(&dn)[8], uint4(&an)[2]) {
    load_d(c, dn);
    load_a(c, an);
  };
  // a set's registers are reloaded only after their last reader (no
  // register copy of a set whose loads are in flight, which would make the
  // compiler wait for them)
  auto step = [&](uint4(&dv)[8], uint4(&av)[2], int next) {
    // column j of the 8 loaded rows
    uint4 frag[8];
    transpose8x8(dv, frag);
    load_d(next, dv);
    lds_barrier();  // previous chunk's readers are done with dt
#pragma unroll
    for (int j = 0; j < 8; ++j) *reinterpret_cast<uint4*>(&dt[(8 * cg + j) * PITCH + 8 * ug]) = frag[j];
    lds_barrier();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8_t A = as_bf16x8(av[ks]);
#pragma unroll
      for (int nf = 0; nf < NF; ++nf) {
        const uint4 bv = *reinterpret_cast<const uint4*>(&dt[(16 * nf + (lane & 15)) * PITCH + 32 * ks + kq]);
        acc[nf] = mfma16(A, as_bf16x8(bv), acc[nf]);
      }
    }
    load_a(next, av);
  };
  const int nc = tk.n_chunks;
  load_chunk(0, d0, a0);
  load_chunk(min(1, nc - 1), d1, a1);
  int c = 0;
  for (; c + 1 < nc; c += 2) {
    step(d0, a0, min(c + 2, nc - 1));
    step(d1, a1, min(c + 3, nc - 1));
  }
  if (c < nc) step(d0, a0, nc - 1);
  // epilogue: fp32 rows of the single partial plane
  float* out = routed ? a.part : a.part_sh + static_cast<size_t>(-1 - tk.expert) * a.sh_plane;
#pragma unroll
  for (int nf = 0; nf < NF; ++nf) {
    const int col = col0 + 16 * nf + (lane & 15);
    if (col < d) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * wave + 4 * (lane >> 4) + r;
        if (row < tr.n) out[static_cast<size_t>(tr.p0 + row) * d + col] = acc[nf][r];
      }
    }
  }
}

// down with both operands staged by direct global -> LDS loads, in the ring
// of the staged gate/up kernel: one stage per chunk (64 units), a work-group
// takes a row tile of up to kGdMaxRows rows (64, 128 or 192 by its rows) x
// kMmaCols columns over all of the expert's chunks.  The down rows of a chunk
// are staged as they sit in memory (unit-major); the B fragments (8 units of
// one column) come out of LDS with transposing reads (ds_read_b64_tr_b16: in
// each 16-lane group, lanes 4 r .. 4 r + 3 give row r of a 4 x 16 tile of
// 16-bit values and lane i receives its column i), two per fragment.  The 16
// byte slots of staged down row u are permuted by 2 (u % 4), so the four
// rows a 16-lane transposing read touches fall in distinct banks.  The waves
// split the tile kGdWaves / 2 x 2: wave (wr, wc) takes the row blocks wr, wr
// + kGdWaves / 2, ... and columns 128 wc .. 128 wc + 127.  The k order of
// every sum (chunks in order, 32 units per MFMA, the same units in the same
// lanes) is that of mma_down_kernel, so the two give the same bits.
constexpr int kDdRowBytes = 2 * kMmaCols;                    // one staged down row
constexpr int kDdBBytes = kChunkUnits * kDdRowBytes;         // the down rows of a stage
static_assert(kGdWaves == 8 && kMmaCols == 256, "wave split of the staged down kernel");

typedef short v4i16_t __attribute__((ext_vector_type(4)));

// 4 x 16 transposing read (see above) at LDS byte address p
__device__ __forceinline__ v4i16_t lds_read_tr16(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16_t*)((const __attribute__((address_space(3))) unsigned char*)(p)));
}

template <int RB>
__device__ __forceinline__ void dd_tile(const MmaArgs& a, const MmaTask& tk, int col0, const TileRows& tr,
                                        unsigned char* lds) {
  constexpr int WR = kGdWaves / 2;                   // row groups of waves
  constexpr int NA = 2 * RB / kGdWaves;              // activation loads per wave and stage
  constexpr int ND = kDdBBytes / kGdLoadBytes / kGdWaves;  // down loads per wave and stage
  constexpr int NL = NA + ND;
  constexpr int HB = RB / WR;                        // row blocks per wave
  constexpr int NF = kMmaCols / 32;                  // column blocks of 16 per wave
  constexpr int ABYTES = RB * kGdBlockBytes;
  constexpr int SBYTES = ABYTES + kDdBBytes;
  constexpr int NST = kGdLds / SBYTES;
  static_assert(RB % WR == 0 && (2 * RB) % kGdWaves == 0 && RB <= kGdMaxRB, "row blocks");
  static_assert(NST >= 2 && (NST - 2) * NL < 64, "ring depth");
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = w >> 1, wc = w & 1;
  const int d = a.d, nc = tk.n_chunks;
  const bool routed = tk.expert >= 0;
  const uint16_t* act = routed ? a.act : a.act_sh + static_cast<size_t>(-1 - tk.expert) * a.rows_shared * a.f_pad_sh;
  const int f_pad = routed ? a.f_pad : a.f_pad_sh;
  // activation loads: as in the gate/up kernel (8 rows of one chunk's 64 units)
  const int lrow = lane >> 3;
  const uint16_t* asrc[NA];
#pragma unroll
  for (int j = 0; j < NA; ++j) {
    const int r = min(8 * (w + kGdWaves * j) + lrow, tr.n - 1);  // rows past the tile repeat its last (never stored)
    asrc[j] = act + static_cast<size_t>(tr.p0 + r) * f_pad + 8 * ((lane & 7) ^ lrow);
  }
  // down loads: 2 rows of 512 bytes each; lane -> row lane / 32, slot lane
  // % 32, which holds piece (lane % 32) ^ (2 (row % 4))
  int doff[ND];
#pragma unroll
  for (int j = 0; j < ND; ++j) {
    const int u = 2 * (w + kGdWaves * j) + (lane >> 5);
    doff[j] = u * d + col0 + 8 * ((lane & 31) ^ (2 * (u & 3)));
  }
  const uint32_t lbase = lds_address(lds) + w * kGdLoadBytes;
  auto issue = [&](int c, int buf) {  // chunks past the last reload it (in bounds, never read)
    c = min(c, nc - 1);
    const uint32_t st = lbase + buf * SBYTES;
#pragma unroll
    for (int j = 0; j < NA; ++j) lds_load16(asrc[j] + c * kChunkUnits, st + kGdWaves * j * kGdLoadBytes);
    const uint16_t* D = reinterpret_cast<const uint16_t*>((c < tk.split ? tk.base : tk.base2) +
                                                          static_cast<size_t>(c) * a.chunk_bytes) +
                        2 * static_cast<size_t>(kChunkUnits) * d;
#pragma unroll
    for (int j = 0; j < ND; ++j) lds_load16(D + doff[j], st + ABYTES + kGdWaves * j * kGdLoadBytes);
  };
  // fragment reads: activations as in the gate/up kernel; down fragments of
  // k step s and column block nf: lane (q = lane / 16, r = lane / 4 % 4, j =
  // lane % 4) reads units 32 s + 8 q + r (+ 4) at columns 16 nf + 4 j .. + 3,
  // whose slot is 16 wc + 2 (nf ^ r) + j / 2 (nf ^ r = 4 (nf / 4) + (nf % 4
  // ^ r))
  int fo[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) fo[s] = (lane & 15) * kGdRowBytes + 16 * ((4 * s + (lane >> 4)) ^ (lane & 7));
  const int tq = lane >> 4, tr4 = (lane >> 2) & 3, tj = lane & 3;
  const int tbase = ABYTES + (8 * tq + tr4) * kDdRowBytes + 16 * (16 * wc + (tj >> 1)) + 8 * (tj & 1);
  int tx[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) tx[b] = tbase + 32 * (b ^ tr4);
  f32x4_t acc[HB][NF];
#pragma unroll
  for (int i = 0; i < HB; ++i)
#pragma unroll
    for (int n = 0; n < NF; ++n) acc[i][n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) {
    const unsigned char* st = lds + buf * SBYTES;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      bf16x8_t B[NF];
#pragma unroll
      for (int n = 0; n < NF; ++n) {
        const unsigned char* p = st + tx[n & 3] + 128 * (n >> 2) + 32 * s * kDdRowBytes;
        const v4i16_t lo = lds_read_tr16(p), hi = lds_read_tr16(p + 4 * kDdRowBytes);
        B[n] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
      const unsigned char* sa = st + wr * kGdBlockBytes + fo[s];
#pragma unroll
      for (int i = 0; i < HB; ++i) {
        const bf16x8_t A = lds_frag(sa + WR * i * kGdBlockBytes);
#pragma unroll
        for (int n = 0; n < NF; ++n) acc[i][n] = mfma16(A, B[n], acc[i][n]);
      }
    }
  };
#pragma unroll
  for (int p = 0; p < NST - 1; ++p) issue(p, p);
  int cur = 0, nxt = NST - 1;
  for (int c = 0; c < nc; ++c) {
    wait_vm<(NST - 2) * NL>();
    bare_barrier();
    issue(c + NST - 1, nxt);
    compute(cur);
    cur = cur + 1 == NST ? 0 : cur + 1;
    nxt = nxt + 1 == NST ? 0 : nxt + 1;
  }
  wait_vm<0>();  // the reloads past the last chunk land before the work-group ends
  float* out = routed ? a.part : a.part_sh + static_cast<size_t>(-1 - tk.expert) * a.sh_plane;
#pragma unroll
  for (int i = 0; i < HB; ++i) {
    const int rb = WR * i + wr;
#pragma unroll
    for (int n = 0; n < NF; ++n) {
      const int col = col0 + 128 * wc + 16 * n + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * rb + 4 * (lane >> 4) + r;
        if (row < tr.n) out[static_cast<size_t>(tr.p0 + row) * d + col] = acc[i][n][r];
      }
    }
  }
}

__global__ __launch_bounds__(64 * kGdWaves) void mma_down_dma_kernel(MmaArgs a) {
  __shared__ __align__(16) unsigned char lds[kGdLds];
  MmaTask tk;
  int local;
  if (!staged_task(a, tk, local)) return;
  const int mt = local / a.ncb, cb = local % a.ncb;
  const TileRows tr = tile_rows(a, tk, mt);
  if (tr.n <= 0) return;  // uniform over the work-group
  if (tr.n <= 64)
    dd_tile<4>(a, tk, cb * kMmaCols, tr, lds);
  else if (tr.n <= 128)
    dd_tile<8>(a, tk, cb * kMmaCols, tr, lds);
  else
    dd_tile<12>(a, tk, cb * kMmaCols, tr, lds);
}

// ------------------------------------------- prefill MFMA over b-bit chunks
//
// The matrix cores take the code pairs as they are: a B fragment of eight
// codes becomes eight bf16 values 1 + q / 2^b (the pair form of the b-bit
// chunk kernel), so an MFMA over one 64-element group yields
// acc = sum_k a_k (1 + q_k / 2^b) and the group adds s (2^b acc - (2^b + z)
// asum) with asum = sum_k a_k of the same rows (one group's accumulator is
// folded in after its two k-steps).  Gate/up: the LDS-staged layout of
// mma_gateup_lds_kernel with each slab's per-row group sums beside it.
// Down: a down column's 64 codes are one group and contiguous, so the B
// fragments load straight from the chunk, without a transpose.

// Code word of elements [kk, kk + 8) of a group (kk a multiple of 8), moved
// so that they form pairs 0 .. 3.
template <int BITS>
__device__ __forceinline__ uint32_t q_word8(const uint32_t* group, int kk) {
  if constexpr (BITS == 2) return group[kk >> 4] >> (kk & 8);  // 16 codes per word: the upper 8 by 8 bits
  else return group[kk >> 3];                                 // 8 codes per word
}

template <int BITS>
__device__ __forceinline__ uint4 q_frag(uint32_t w, const PairMasks<BITS>& pm) {
  return make_uint4(code_pair<BITS, 0>(w, pm), code_pair<BITS, 1>(w, pm), code_pair<BITS, 2>(w, pm),
                    code_pair<BITS, 3>(w, pm));
}

template <int BITS>
__global__ __launch_bounds__(256) void mma_gateup_q_kernel(MmaArgs a) {
  __shared__ __align__(16) uint16_t As[2][kMmaRows * kGuPitch];
  __shared__ float asum[2][kMmaRows][2];  // per slab buffer: [row][group of the slab]
  constexpr float C = static_cast<float>(1 << BITS);
  constexpr int GW = 2 * BITS;  // code words per group
  const PairMasks<BITS> pm;
  const int wg = xcd_local(blockIdx.x, gridDim.x);
  const MmaTask tk = a.tasks[find_task(a.tasks, a.n_tasks, wg)];
  const int local = wg - tk.wg_begin;
  const int mt = local % tk.m_tiles;
  const int c = tk.chunk_lo + local / tk.m_tiles;
  const TileRows tr = tile_rows(a, tk, mt);
  if (tr.n <= 0) return;  // uniform over the work-group
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d, ngr = d / 64;
  const int ksteps = d / 32;
  const int nslab = (ksteps + 3) / 4;
  const uint16_t* hrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = min((tid >> 4) + 16 * i, tr.n - 1);  // clamped rows: staged, never stored
    const int tok = a.perm[tr.p0 + row] / a.K;  // b-bit experts are routed only
    hrow[i] = static_cast<const uint16_t*>(a.h) + static_cast<size_t>(tok) * d + 8 * (tid & 15);
  }
  const unsigned char* chunk = tk.base + static_cast<size_t>(c) * a.chunk_bytes;
  const size_t qrow = static_cast<size_t>(d) * BITS / 8;
  const uint32_t* Gq = reinterpret_cast<const uint32_t*>(chunk);
  const uint32_t* Uq = reinterpret_cast<const uint32_t*>(chunk + 64 * qrow);
  const uint32_t* Gm = reinterpret_cast<const uint32_t*>(chunk + 192 * qrow);
  const uint32_t* Um = Gm + 64 * ngr;
  const int unit = 16 * wave + (lane & 15);
  const int kq = 8 * (lane >> 4);
  uint4 ast[4];
  // per slab: two groups x (k-step words of G and U) + the groups' metadata
  uint32_t gw[2][2], uw[2][2], gmn[2], umn[2];
  uint32_t gwc[2][2], uwc[2][2], gmc[2], umc[2];
  auto load_a = [&](int sl) {
    const int k0 = min(sl, nslab - 1) * kGuSlab;
#pragma unroll
    for (int i = 0; i < 4; ++i) ast[i] = ld16(hrow[i] + min(k0, d - kGuSlab));
  };
  auto store_a = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<uint4*>(&As[buf][((tid >> 4) + 16 * i) * kGuPitch + 8 * (tid & 15)]) = ast[i];
  };
  auto load_b = [&](int sl) {
#pragma unroll
    for (int gi = 0; gi < 2; ++gi) {
      const int g = min(2 * sl + gi, ngr - 1);  // clamped past the last group (loaded, not used)
      const uint32_t* gq = Gq + (static_cast<size_t>(unit) * ngr + g) * GW;
      const uint32_t* uq = Uq + (static_cast<size_t>(unit) * ngr + g) * GW;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        gw[gi][s] = q_word8<BITS>(gq, 32 * s + kq);
        uw[gi][s] = q_word8<BITS>(uq, 32 * s + kq);
      }
      gmn[gi] = Gm[static_cast<size_t>(unit) * ngr + g];
      umn[gi] = Um[static_cast<size_t>(unit) * ngr + g];
    }
  };
  // per-row sums of the staged slab's two 64-wide groups (window-relative)
  auto row_sums = [&](int buf) {
    if (tid < 2 * kMmaRows) {
      const int row = tid >> 1, gi = tid & 1;
      const uint4* src = reinterpret_cast<const uint4*>(&As[buf][row * kGuPitch + 64 * gi]);
      float sum = 0.0f;
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const uint4 x = src[v];
        sum = dot2bf(x.x, kBf16OnePair, sum);
        sum = dot2bf(x.y, kBf16OnePair, sum);
        sum = dot2bf(x.z, kBf16OnePair, sum);
        sum = dot2bf(x.w, kBf16OnePair, sum);
      }
      asum[buf][row][gi] = sum;
    }
  };
  f32x4_t ag[4], au[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) ag[rb] = au[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  load_a(0);
  load_b(0);
  store_a(0);
  __syncthreads();
  row_sums(0);
  __syncthreads();
  for (int sl = 0; sl < nslab; ++sl) {
    const int buf = sl & 1;
#pragma unroll
    for (int gi = 0; gi < 2; ++gi) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        gwc[gi][s] = gw[gi][s];
        uwc[gi][s] = uw[gi][s];
      }
      gmc[gi] = gmn[gi];
      umc[gi] = umn[gi];
    }
    load_a(sl + 1);
    load_b(sl + 1);
    const int k0 = sl * kGuSlab, kbase = k0 - min(k0, d - kGuSlab);  // a partial last slab sits at the window's end
#pragma unroll
    for (int gi = 0; gi < 2; ++gi) {
      if (2 * sl + gi < ngr) {
        const int wgi = (kbase >> 6) + gi;  // the group's half of the staged window
        const float gs = fp16_lo(gmc[gi]), gz = C + fp16_hi(gmc[gi]);
        const float us = fp16_lo(umc[gi]), uz = C + fp16_hi(umc[gi]);
        const uint4 bg0 = q_frag<BITS>(gwc[gi][0], pm), bg1 = q_frag<BITS>(gwc[gi][1], pm);
        const uint4 bu0 = q_frag<BITS>(uwc[gi][0], pm), bu1 = q_frag<BITS>(uwc[gi][1], pm);
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
          if (16 * rb < tr.n) {
            const uint16_t* ar = &As[buf][(16 * rb + (lane & 15)) * kGuPitch + 64 * wgi + kq];
            const bf16x8_t A0 = as_bf16x8(*reinterpret_cast<const uint4*>(ar));
            const bf16x8_t A1 = as_bf16x8(*reinterpret_cast<const uint4*>(ar + 32));
            f32x4_t cg = mfma16(A0, as_bf16x8(bg0), f32x4_t{0.f, 0.f, 0.f, 0.f});
            cg = mfma16(A1, as_bf16x8(bg1), cg);
            f32x4_t cu = mfma16(A0, as_bf16x8(bu0), f32x4_t{0.f, 0.f, 0.f, 0.f});
            cu = mfma16(A1, as_bf16x8(bu1), cu);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float xs = asum[buf][16 * rb + 4 * (lane >> 4) + r][wgi];
              ag[rb][r] += gs * (C * cg[r] - gz * xs);
              au[rb][r] += us * (C * cu[r] - uz * xs);
            }
          }
        }
      }
    }
    if (sl + 1 < nslab) {
      store_a(buf ^ 1);
      __syncthreads();
      row_sums(buf ^ 1);
    }
    __syncthreads();
  }
  uint16_t* act = a.act;  // b-bit experts are routed only
  const int f = c * kChunkUnits + unit;
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 16 * rb + 4 * (lane >> 4) + r;
      if (row < tr.n) act[static_cast<size_t>(tr.p0 + row) * a.f_pad + f] = f2bf(silu(ag[rb][r]) * au[rb][r]);
    }
  }
}

template <int BITS>
__global__ __launch_bounds__(256) void mma_down_q_kernel(MmaArgs a) {
  constexpr float C = static_cast<float>(1 << BITS);
  constexpr int GW = 2 * BITS;  // code words per column group
  constexpr int NF = kMmaCols / 16;
  const PairMasks<BITS> pm;
  const int wg = xcd_local(blockIdx.x, gridDim.x);
  const MmaTask tk = a.tasks[find_task(a.tasks, a.n_tasks, wg)];
  const int local = wg - tk.wg_begin;
  // work-group = (row tile, column block, chunk range): ranges of
  // ceil(n_chunks / ksplit) chunks, range ks summed into plane ks
  const int ks = local % a.ksplit;
  const int mt = (local / a.ksplit) / a.ncb, cb = (local / a.ksplit) % a.ncb;
  const TileRows tr = tile_rows(a, tk, mt);
  if (tr.n <= 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (16 * wave >= tr.n) return;  // no rows for this wave (no barrier in this kernel)
  const int d = a.d;
  const size_t qrow = static_cast<size_t>(d) * BITS / 8;
  const int ar = min(16 * wave + (lane & 15), tr.n - 1);
  const uint16_t* arow = a.act + static_cast<size_t>(tr.p0 + ar) * a.f_pad;
  const int kq = 8 * (lane >> 4);
  const int col0 = cb * kMmaCols;
  f32x4_t acc[NF];
#pragma unroll
  for (int nf = 0; nf < NF; ++nf) acc[nf] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // one chunk: the A fragments of its 64 units, and per column block this
  // lane's two code words and the column's metadata
  uint4 an[2], ac[2];
  uint32_t wn[NF][2], mn[NF], wc[NF][2], mc[NF];
  auto load_chunk = [&](int cc) {
    const unsigned char* cbase = (cc < tk.split ? tk.base : tk.base2) + static_cast<size_t>(cc) * a.chunk_bytes;
    const uint32_t* Dq = reinterpret_cast<const uint32_t*>(cbase + 128 * qrow);
    const uint32_t* Dm = reinterpret_cast<const uint32_t*>(cbase + 192 * qrow) + 128 * (d / 64);
#pragma unroll
    for (int nf = 0; nf < NF; ++nf) {
      const int col = min(col0 + 16 * nf + (lane & 15), d - 1);  // clamped; columns past d are never stored
      const uint32_t* grp = Dq + static_cast<size_t>(col) * GW;
      wn[nf][0] = q_word8<BITS>(grp, kq);
      wn[nf][1] = q_word8<BITS>(grp, 32 + kq);
      mn[nf] = Dm[col];
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) an[ks] = ld16(arow + cc * kChunkUnits + 32 * ks + kq);
  };
  const int per = (tk.n_chunks + a.ksplit - 1) / a.ksplit;
  const int c_lo = min(ks * per, tk.n_chunks), nc = min(tk.n_chunks, c_lo + per);
  load_chunk(min(c_lo, tk.n_chunks - 1));  // an empty range loads (in bounds) and computes nothing
  for (int cc = c_lo; cc < nc; ++cc) {
#pragma unroll
    for (int nf = 0; nf < NF; ++nf) {
      wc[nf][0] = wn[nf][0];
      wc[nf][1] = wn[nf][1];
      mc[nf] = mn[nf];
    }
    ac[0] = an[0];
    ac[1] = an[1];
    load_chunk(min(cc + 1, nc - 1));  // the last chunk reloads itself (in bounds, unused)
    // the chunk's activation sum of each row: this lane's 16 values, then the
    // four lanes of the row; rows of the result layout come from lane row
    float xs = 0.0f;
    const uint32_t av[8] = {ac[0].x, ac[0].y, ac[0].z, ac[0].w, ac[1].x, ac[1].y, ac[1].z, ac[1].w};
#pragma unroll
    for (int i = 0; i < 8; ++i) xs = dot2bf(av[i], kBf16OnePair, xs);
    xs += __shfl_xor(xs, 16, 64);
    xs += __shfl_xor(xs, 32, 64);
    float rs[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) rs[r] = __shfl(xs, 4 * (lane >> 4) + r, 64);
    const bf16x8_t A0 = as_bf16x8(ac[0]), A1 = as_bf16x8(ac[1]);
#pragma unroll
    for (int nf = 0; nf < NF; ++nf) {
      f32x4_t cacc = mfma16(A0, as_bf16x8(q_frag<BITS>(wc[nf][0], pm)), f32x4_t{0.f, 0.f, 0.f, 0.f});
      cacc = mfma16(A1, as_bf16x8(q_frag<BITS>(wc[nf][1], pm)), cacc);
      const float s = fp16_lo(mc[nf]), z = C + fp16_hi(mc[nf]);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[nf][r] += s * (C * cacc[r] - z * rs[r]);
    }
  }
#pragma unroll
  for (int nf = 0; nf < NF; ++nf) {
    const int col = col0 + 16 * nf + (lane & 15);
    if (col < d) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * wave + 4 * (lane >> 4) + r;
        if (row < tr.n) a.part[(static_cast<size_t>(tr.p0 + row) * a.ksplit + ks) * d + col] = acc[nf][r];
      }
    }
  }
}

// Prefill plan (see launch_prefill_plan): thread i takes routed expert i,
// or shared expert i - E; exclusive scans over the threads give each task
// its index and first work-group.
__global__ __launch_bounds__(kMaxPlanTasks) void prefill_plan_kernel(PlanArgs p) {
  __shared__ int4 sc[2][kMaxPlanTasks];
  const int i = threadIdx.x;
  MmaTask t{};
  int gu_w = 0, dn_w = 0, gu_c = 0, dn_c = 0;
  if (i < p.E) {
    const int n = p.offsets[i + 1] - p.offsets[i];
    const int res = p.res[i];
    if (n > 0 && res > 0) {
      t.base = p.cache_base + p.top_bytes * static_cast<uint64_t>(p.slot[i]);
      t.expert = i;
      t.m_tiles = (n + p.tile_rows - 1) / p.tile_rows;
      gu_c = res;
      gu_w = t.m_tiles * ((res + gd_group_chunks(n, res) - 1) / gd_group_chunks(n, res));
      if (res >= p.n_chunks) {
        dn_c = p.n_chunks;
        dn_w = t.m_tiles * p.ncb;
      }
    }
  } else if (i < p.E + p.n_sh && p.T > 0) {
    const int sh = i - p.E;
    t.base = p.shared[sh];
    t.expert = -1 - sh;
    t.m_tiles = (p.T + p.tile_rows - 1) / p.tile_rows;
    gu_c = dn_c = p.n_chunks_sh;
    gu_w = t.m_tiles * ((p.n_chunks_sh + gd_group_chunks(p.T, p.n_chunks_sh) - 1) / gd_group_chunks(p.T, p.n_chunks_sh));
    dn_w = t.m_tiles * p.ncb;
  }
  // inclusive scan of (gate/up task, gate/up work-groups, down task, down work-groups)
  int4 v = make_int4(gu_w > 0, gu_w, dn_w > 0, dn_w);
  int cur = 0;
  sc[0][i] = v;
  __syncthreads();
  for (int off = 1; off < kMaxPlanTasks; off <<= 1) {
    if (i >= off) {
      const int4 o = sc[cur][i - off];
      v = make_int4(v.x + o.x, v.y + o.y, v.z + o.z, v.w + o.w);
    }
    sc[cur ^ 1][i] = v;
    cur ^= 1;
    __syncthreads();
  }
  t.base2 = t.base;
  if (gu_w > 0) {
    MmaTask g = t;
    g.n_chunks = gu_c;
    g.wg_begin = v.y - gu_w;
    p.gu[v.x - 1] = g;
  }
  if (dn_w > 0) {
    MmaTask g = t;
    g.n_chunks = dn_c;
    g.split = dn_c;  // every chunk from base
    g.wg_begin = v.w - dn_w;
    p.dn[v.z - 1] = g;
  }
  if (i == kMaxPlanTasks - 1) {
    p.counts[0] = v.x;
    p.counts[1] = v.y;
    p.counts[2] = v.z;
    p.counts[3] = v.w;
  }
}

hipError_t launch_prefill_plan(const PlanArgs& a, hipStream_t s) {
  if (a.E < 0 || a.n_sh < 0 || a.n_sh > kMaxPlanShared || a.E + a.n_sh > kMaxPlanTasks || a.tile_rows <= 0)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(prefill_plan_kernel, dim3(1), dim3(kMaxPlanTasks), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mma_gateup(const MmaArgs& a, hipStream_t s) {
  if (a.dtasks) {
    if (a.n_wg <= 0) return hipSuccess;
    if (a.bits != 0 || a.gu_split != 1 || a.d % (2 * kGdSlab) != 0 || a.tile_rows > kGdMaxRows || !a.dcount)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(mma_gateup_dma_kernel, dim3(a.n_wg), dim3(64 * kGdWaves), 0, s, a);
    return hipGetLastError();
  }
  if (a.n_wg <= 0 || a.n_tasks <= 0) return hipSuccess;
  if (a.bits != 0) {
    if (a.gu_split != 1 || !q_supported(a.d)) return hipErrorInvalidValue;
    if (a.bits == 2)
      hipLaunchKernelGGL(mma_gateup_q_kernel<2>, dim3(a.n_wg), dim3(256), 0, s, a);
    else if (a.bits == 4)
      hipLaunchKernelGGL(mma_gateup_q_kernel<4>, dim3(a.n_wg), dim3(256), 0, s, a);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (a.gu_split == 4)
    hipLaunchKernelGGL(mma_gateup_kernel<1>, dim3(a.n_wg), dim3(256), kGuardLds, s, a);
  else if (a.gu_split == 1 && a.d % (2 * kGdSlab) == 0 && a.tile_rows <= kGdMaxRows)
    hipLaunchKernelGGL(mma_gateup_dma_kernel, dim3(a.n_wg), dim3(64 * kGdWaves), 0, s, a);
  else if (a.gu_split == 1 && a.tile_rows == kMmaRows)
    hipLaunchKernelGGL(mma_gateup_kernel<4>, dim3(a.n_wg), dim3(256), kGuardLds, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_mma_down(const MmaArgs& a, hipStream_t s) {
  if (a.dtasks) {
    if (a.n_wg <= 0) return hipSuccess;
    if (a.bits != 0 || a.ksplit != 1 || a.d % kMmaCols != 0 || a.tile_rows != kGdMaxRows || !a.dcount)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(mma_down_dma_kernel, dim3(a.n_wg), dim3(64 * kGdWaves), 0, s, a);
    return hipGetLastError();
  }
  if (a.n_wg <= 0 || a.n_tasks <= 0) return hipSuccess;
  if (a.ksplit < 1 || (a.bits == 0 && a.ksplit != 1)) return hipErrorInvalidValue;
  if (a.bits != 0) {
    if (!q_supported(a.d)) return hipErrorInvalidValue;
    if (a.bits == 2)
      hipLaunchKernelGGL(mma_down_q_kernel<2>, dim3(a.n_wg), dim3(256), kGuardLds, s, a);
    else if (a.bits == 4)
      hipLaunchKernelGGL(mma_down_q_kernel<4>, dim3(a.n_wg), dim3(256), kGuardLds, s, a);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (a.tile_rows == kGdMaxRows && a.d % kMmaCols == 0)
    hipLaunchKernelGGL(mma_down_dma_kernel, dim3(a.n_wg), dim3(64 * kGdWaves), 0, s, a);
  else if (a.tile_rows == kMmaRows)
    hipLaunchKernelGGL(mma_down_kernel, dim3(a.n_wg), dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// ------------------------------------------------------ residual + RMSNorm
//
// 256 threads per token; each holds up to kRnPer 16-byte pieces of the row
// (d <= 8192).  Squares are summed per thread, then over the wave with a
// butterfly and over the four waves in order.

constexpr int kRnThreads = 256;

template <typename W>
__global__ __launch_bounds__(kRnThreads) void residual_norm_kernel(const W* __restrict__ h,
                                                                   const float* __restrict__ y,
                                                                   W* __restrict__ out, int d, float eps) {
  constexpr int VEC = Vec<W>::N;
  constexpr int PER = kMaxModelDim / (kRnThreads * VEC);  // 16-byte pieces per thread at most
  __shared__ float wsum[kRnThreads / 64];
  const int t = blockIdx.x, tid = threadIdx.x;
  const W* hr = h + static_cast<size_t>(t) * d;
  const float* yr = y + static_cast<size_t>(t) * d;
  W* orow = out + static_cast<size_t>(t) * d;
  const int n = d / VEC;  // 16-byte pieces of the row
  float x[PER][VEC];
  float ss = 0.0f;
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int i = tid + m * kRnThreads;
    if (i < n) {
      float hv[VEC];
      unpack(ld16(hr + static_cast<size_t>(i) * VEC), hv);
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        x[m][j] = hv[j] + yr[static_cast<size_t>(i) * VEC + j];
        ss = fmaf(x[m][j], x[m][j], ss);
      }
    }
  }
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) ss += __shfl_xor(ss, s, 64);
  if ((tid & 63) == 0) wsum[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < kRnThreads / 64; ++w) tot += wsum[w];
  const float inv = 1.0f / sqrtf(tot / static_cast<float>(d) + eps);
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int i = tid + m * kRnThreads;
    if (i < n) {
      if constexpr (sizeof(W) == 2) {
        uint32_t wv[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          wv[j] = static_cast<uint32_t>(f2bf(x[m][2 * j] * inv)) | (static_cast<uint32_t>(f2bf(x[m][2 * j + 1] * inv)) << 16);
        *reinterpret_cast<uint4*>(orow + static_cast<size_t>(i) * VEC) = make_uint4(wv[0], wv[1], wv[2], wv[3]);
      } else {
        *reinterpret_cast<float4*>(orow + static_cast<size_t>(i) * VEC) =
            make_float4(x[m][0] * inv, x[m][1] * inv, x[m][2] * inv, x[m][3] * inv);
      }
    }
  }
}

hipError_t launch_residual_norm(const void* h, const float* y, void* out, int T, int d, int dtype, float eps,
                                hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (d <= 0 || d > kMaxModelDim || d % 64 != 0) return hipErrorInvalidValue;
  if (dtype == kBF16)
    hipLaunchKernelGGL(residual_norm_kernel<uint16_t>, dim3(T), dim3(kRnThreads), 0, s,
                       static_cast<const uint16_t*>(h), y, static_cast<uint16_t*>(out), d, eps);
  else
    hipLaunchKernelGGL(residual_norm_kernel<float>, dim3(T), dim3(kRnThreads), 0, s, static_cast<const float*>(h), y,
                       static_cast<float*>(out), d, eps);
  return hipGetLastError();
}

// --------------------------------------------------------------- H2D copy
//
// Each work-group moves NTH x kH2dUnroll 16-byte pieces per round (all loads
// of a round issued before its stores), rounds strided over the grid.  The
// host copy's 16 work-groups of 512 threads keep enough PCIe reads in flight
// to reach the link rate; each holds its CU's LDS (never touched: the
// allocation alone keeps other work-groups that request LDS off the CU).

constexpr int kH2dUnroll = 4;

template <int NTH, bool HOLD_CU>
__global__ __launch_bounds__(NTH) void copy_kernel(uint4* __restrict__ dst, const uint4* __restrict__ src,
                                                   uint64_t n) {
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * NTH * kH2dUnroll;
  for (uint64_t base = static_cast<uint64_t>(blockIdx.x) * NTH * kH2dUnroll + threadIdx.x; base < n;
       base += stride) {
    uint4 v[kH2dUnroll];
#pragma unroll
    for (int u = 0; u < kH2dUnroll; ++u) {
      const uint64_t i = base + static_cast<uint64_t>(u) * NTH;
      v[u] = src[i < n ? i : n - 1];  // clamped: every load is issued and in bounds
    }
#pragma unroll
    for (int u = 0; u < kH2dUnroll; ++u) {
      const uint64_t i = base + static_cast<uint64_t>(u) * NTH;
      if (i < n) dst[i] = v[u];
    }
  }
  if constexpr (HOLD_CU) {
    __shared__ uint4 hold[kCuLdsBytes / 16];
    if (n == 0) {  // the host never launches an empty copy: keeps the allocation, never runs
      hold[threadIdx.x] = make_uint4(0, 0, 0, 0);
      __syncthreads();
      dst[0] = hold[(threadIdx.x + 1) % NTH];
    }
  }
}

template <int NTH, bool HOLD_CU>
static hipError_t launch_copy(void* dst, const void* src, uint64_t bytes, int max_wgs, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  if ((bytes % 16) != 0 || (reinterpret_cast<uintptr_t>(dst) % 16) != 0 || (reinterpret_cast<uintptr_t>(src) % 16) != 0)
    return hipErrorInvalidValue;
  const uint64_t n = bytes / 16;
  const uint64_t per_wg = static_cast<uint64_t>(NTH) * kH2dUnroll;
  const int wgs = static_cast<int>(std::min<uint64_t>(max_wgs, (n + per_wg - 1) / per_wg));
  hipLaunchKernelGGL((copy_kernel<NTH, HOLD_CU>), dim3(wgs), dim3(NTH), 0, s, static_cast<uint4*>(dst),
                     static_cast<const uint4*>(src), n);
  return hipGetLastError();
}

hipError_t launch_h2d(void* dst, const void* src, uint64_t bytes, hipStream_t s) {
  return launch_copy<kH2dThreads, true>(dst, src, bytes, kH2dWorkGroups, s);
}

hipError_t launch_d2d(void* dst, const void* src, uint64_t bytes, hipStream_t s) {
  return launch_copy<256, false>(dst, src, bytes, kD2dWorkGroups, s);
}

// ------------------------------------------------------------------ combine
//
// The partial planes are summed in a fixed order, so the output is the same
// whichever stream or launch produced each plane.  More than kCombFewTokens
// tokens: two launches,
//  1. work-group (term slot, 256 columns, plane group g): wave w sums planes
//     p = 4 g + w + 4 G j (j ascending, four interleaved accumulators added
//     in order); the four wave sums are added in wave order -> red[g][slot];
//  2. per (token, 256 columns): S_term = sum_g red[g][slot] (g ascending),
//     y[t] = sum_k w[t][k] * S_k in selection order, then + the shared
//     experts' S_s in index order.

constexpr int kCombWaves = 4;
constexpr int kCombMaxGroups = 16;

__device__ __forceinline__ float4 f4add(float4 x, float4 y) {
  return make_float4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
}

__global__ __launch_bounds__(64 * kCombWaves) void combine_planes_kernel(CombineArgs a) {
  __shared__ float4 red4[kCombWaves][64];
  const int ts = blockIdx.x, cb = blockIdx.y, pg = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = cb * 256 + lane * 4;
  const bool live = col < a.d;
  const int TK = a.T * a.K;
  const int n_slots = TK + a.T * a.n_shared;
  const float* base;
  int row, np;
  if (ts < TK) {
    base = a.part;
    row = a.pos[ts];
    np = a.n_planes;
  } else {
    const int si = ts - TK;
    const int t = si / a.n_shared;
    const int sh = si - t * a.n_shared;
    base = a.part_sh + static_cast<size_t>(sh) * a.sh_plane;
    row = t;
    np = a.n_planes_sh;
  }
  float4 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (live) {
    const float* rbase = base + static_cast<size_t>(row) * np * a.d + col;  // this slot's contiguous planes
    const int stride = kCombWaves * a.pg;
    for (int p0 = pg * kCombWaves + wave; p0 < np; p0 += 4 * stride) {
      float4 v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)  // clamped loads, unused ones dropped below
        v[i] = *reinterpret_cast<const float4*>(rbase + static_cast<size_t>(min(p0 + i * stride, np - 1)) * a.d);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (p0 + i * stride < np) acc[i] = f4add(acc[i], v[i]);
    }
  }
  red4[wave][lane] = f4add(f4add(acc[0], acc[1]), f4add(acc[2], acc[3]));
  __syncthreads();
  if (wave == 0 && live) {
    float4 tot = red4[0][lane];
    for (int w2 = 1; w2 < kCombWaves; ++w2) tot = f4add(tot, red4[w2][lane]);
    *reinterpret_cast<float4*>(a.red + (static_cast<size_t>(pg) * n_slots + ts) * a.d + col) = tot;
  }
}

// The loads of up to 16 (term, group) partial sums are in flight at once:
// PG groups of 16 / PG terms.
template <int PG>
__global__ __launch_bounds__(64) void combine_final_kernel(CombineArgs a) {
  constexpr int TB = PG >= 16 ? 1 : 16 / PG;  // terms per batch
  const int t = blockIdx.x;
  const int col = blockIdx.y * 256 + threadIdx.x * 4;
  if (col >= a.d) return;
  const int TK = a.T * a.K;
  const int n_slots = TK + a.T * a.n_shared;
  const int n_terms = a.K + a.n_shared;
  float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k0 = 0; k0 < n_terms; k0 += TB) {
    float4 v[TB][PG];
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      const int term = min(k0 + j, n_terms - 1);  // clamped: in bounds, used only in range
      const int slot = term < a.K ? t * a.K + term : TK + t * a.n_shared + (term - a.K);
#pragma unroll
      for (int g = 0; g < PG; ++g)
        v[j][g] = *reinterpret_cast<const float4*>(a.red + (static_cast<size_t>(g) * n_slots + slot) * a.d + col);
    }
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      const int term = k0 + j;
      if (term < n_terms) {
        float4 sum = v[j][0];
#pragma unroll
        for (int g = 1; g < PG; ++g) sum = f4add(sum, v[j][g]);
        if (term < a.K) {
          const float wk = a.w[t * a.K + term];
          y = make_float4(fmaf(wk, sum.x, y.x), fmaf(wk, sum.y, y.y), fmaf(wk, sum.z, y.z), fmaf(wk, sum.w, y.w));
        } else {
          y = f4add(y, sum);
        }
      }
    }
  }
  *reinterpret_cast<float4*>(a.y + static_cast<size_t>(t) * a.d + col) = y;
}

// Few tokens (T <= kCombFewTokens): one launch.  Work-group (32 columns,
// token t); thread (plane lane pl = tid / 8, column quad tid % 8).  Per term
// (the token's K routed slots in selection order, then its shared experts):
// the thread sums planes pl, pl + 32, ... in order; the 8 plane lanes of a
// wave are added by an xor butterfly over lane bits 3..5; the 4 wave sums
// are added as (w0 + w1) + (w2 + w3).  Then y[t] = sum_k w[t][k] * S_k in
// selection order, plus the shared experts' S_s in index order.  A thread
// keeps 16 plane loads in flight: PER planes of each of 16 / PER terms.
constexpr int kCombFewTokens = 8;
constexpr int kCombCols = 32;  // columns per work-group
constexpr int kCombMaxTerms = kMaxTopK + 8;

__device__ __forceinline__ void comb_term(const CombineArgs& a, int t, int term, const float*& rbase, int& np) {
  if (term < a.K) {
    const int row = a.pos[t * a.K + term];
    rbase = a.part + static_cast<size_t>(row) * a.n_planes * a.d;
    np = a.n_planes;
  } else {
    const int sh = term - a.K;
    rbase = a.part_sh + static_cast<size_t>(sh) * a.sh_plane + static_cast<size_t>(t) * a.n_planes_sh * a.d;
    np = a.n_planes_sh;
  }
}

template <int PER>
__global__ __launch_bounds__(256) void combine_few_kernel(CombineArgs a) {
  constexpr int TPB = 16 / PER;  // terms per batch
  __shared__ float4 red[kCombMaxTerms][4][kCombCols / 4];
  __shared__ float w_s[kMaxTopK];
  const int t = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cq = tid & 7, pl = tid >> 3;  // plane lane 0..31
  const int col = blockIdx.x * kCombCols + 4 * cq;
  const bool live = col < a.d;
  const int n_terms = a.K + a.n_shared;
  // the token's weights, requested with the first partial loads (read after
  // the barrier)
  if (tid < a.K) w_s[tid] = a.w[t * a.K + tid];
  for (int k0 = 0; k0 < n_terms; k0 += TPB) {
    const float* rb[TPB];
    int np[TPB];
    int np_max = 0;
#pragma unroll
    for (int j = 0; j < TPB; ++j) {
      rb[j] = a.part;
      np[j] = 0;
      if (k0 + j < n_terms) comb_term(a, t, k0 + j, rb[j], np[j]);
      np_max = max(np_max, np[j]);
    }
    float4 acc[TPB];
#pragma unroll
    for (int j = 0; j < TPB; ++j) acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int p0 = pl; p0 < np_max; p0 += 32 * PER) {
      float4 v[TPB][PER];
#pragma unroll
      for (int j = 0; j < TPB; ++j)
#pragma unroll
        for (int i = 0; i < PER; ++i) {
          const int p = min(p0 + 32 * i, np[j] - 1);  // clamped: in bounds, used only in range
          v[j][i] = (live && np[j] > 0) ? *reinterpret_cast<const float4*>(rb[j] + static_cast<size_t>(p) * a.d + col)
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
      for (int j = 0; j < TPB; ++j)
#pragma unroll
        for (int i = 0; i < PER; ++i)
          if (p0 + 32 * i < np[j]) acc[j] = f4add(acc[j], v[j][i]);
    }
#pragma unroll
    for (int j = 0; j < TPB; ++j) {
      if (k0 + j >= n_terms) continue;  // the same for the whole work-group
#pragma unroll
      for (int m = 8; m <= 32; m <<= 1) {
        float4 o;
        o.x = __shfl_xor(acc[j].x, m, 64);
        o.y = __shfl_xor(acc[j].y, m, 64);
        o.z = __shfl_xor(acc[j].z, m, 64);
        o.w = __shfl_xor(acc[j].w, m, 64);
        acc[j] = f4add(acc[j], o);
      }
      if (lane < 8) red[k0 + j][wave][cq] = acc[j];
    }
  }
  __syncthreads();
  if (tid < 8 && live) {
    float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int term = 0; term < n_terms; ++term) {
      const float4 sum = f4add(f4add(red[term][0][cq], red[term][1][cq]), f4add(red[term][2][cq], red[term][3][cq]));
      if (term < a.K) {
        const float wk = w_s[term];
        y = make_float4(fmaf(wk, sum.x, y.x), fmaf(wk, sum.y, y.y), fmaf(wk, sum.z, y.z), fmaf(wk, sum.w, y.w));
      } else {
        y = f4add(y, sum);
      }
    }
    *reinterpret_cast<float4*>(a.y + static_cast<size_t>(t) * a.d + col) = y;
  }
}

// One partial plane per slot (prefill path): the same sums in one pass,
// straight from the partials (a first pass would only copy them).
__global__ __launch_bounds__(64) void combine_direct_kernel(CombineArgs a) {
  const int t = blockIdx.x;
  const int col = blockIdx.y * 256 + threadIdx.x * 4;
  if (col >= a.d) return;
  float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
  // routed terms in batches of kDirectBatch: their rows, then their partial
  // loads, all in flight before the first is added (the order of the sum is
  // the terms' order)
  constexpr int kDirectBatch = 8;
  for (int k0 = 0; k0 < a.K; k0 += kDirectBatch) {
    int row[kDirectBatch];
    float wk[kDirectBatch];
#pragma unroll
    for (int j = 0; j < kDirectBatch; ++j) {
      const int k = min(k0 + j, a.K - 1);  // clamped: in bounds, used only below K
      row[j] = a.pos[t * a.K + k];
      wk[j] = a.w[t * a.K + k];
    }
    float4 v[kDirectBatch];
#pragma unroll
    for (int j = 0; j < kDirectBatch; ++j)
      v[j] = *reinterpret_cast<const float4*>(a.part + static_cast<size_t>(row[j]) * a.d + col);
#pragma unroll
    for (int j = 0; j < kDirectBatch; ++j)
      if (k0 + j < a.K)
        y = make_float4(fmaf(wk[j], v[j].x, y.x), fmaf(wk[j], v[j].y, y.y), fmaf(wk[j], v[j].z, y.z),
                        fmaf(wk[j], v[j].w, y.w));
  }
  for (int sh = 0; sh < a.n_shared; ++sh)
    y = f4add(y, *reinterpret_cast<const float4*>(a.part_sh + static_cast<size_t>(sh) * a.sh_plane +
                                                  static_cast<size_t>(t) * a.d + col));
  *reinterpret_cast<float4*>(a.y + static_cast<size_t>(t) * a.d + col) = y;
}

int combine_groups(int T, int K, int n_shared, int d, int n_planes) {
  const int slots = T * (K + n_shared);
  const int ncb = (d + 255) / 256;
  int g = 1;
  while (g < kCombMaxGroups && static_cast<int64_t>(slots) * ncb * g * 2 <= 512 && g * 2 * kCombWaves <= n_planes)
    g *= 2;
  return g;
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  const int ncb = (a.d + 255) / 256;
  if (a.n_planes == 1 && (a.n_shared == 0 || a.n_planes_sh == 1)) {
    hipLaunchKernelGGL(combine_direct_kernel, dim3(a.T, ncb), dim3(64), kGuardLds, s, a);
    return hipGetLastError();
  }
  if (a.T <= kCombFewTokens && a.K + a.n_shared <= kCombMaxTerms) {
    const dim3 grid((a.d + kCombCols - 1) / kCombCols, a.T);
    const int per = (std::max(a.n_planes, a.n_shared > 0 ? a.n_planes_sh : 0) + 31) / 32;
    if (per <= 1)
      hipLaunchKernelGGL(combine_few_kernel<1>, grid, dim3(256), 0, s, a);
    else if (per <= 2)
      hipLaunchKernelGGL(combine_few_kernel<2>, grid, dim3(256), 0, s, a);
    else if (per <= 4)
      hipLaunchKernelGGL(combine_few_kernel<4>, grid, dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL(combine_few_kernel<8>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const int slots = a.T * (a.K + a.n_shared);
  hipLaunchKernelGGL(combine_planes_kernel, dim3(slots, ncb, a.pg), dim3(64 * kCombWaves), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  auto* fin = a.pg == 1   ? combine_final_kernel<1>
              : a.pg == 2 ? combine_final_kernel<2>
              : a.pg == 4 ? combine_final_kernel<4>
              : a.pg == 8 ? combine_final_kernel<8>
                          : combine_final_kernel<16>;
  hipLaunchKernelGGL(fin, dim3(a.T, ncb), dim3(64), kGuardLds, s, a);
  return hipGetLastError();
}

}  // namespace msk
