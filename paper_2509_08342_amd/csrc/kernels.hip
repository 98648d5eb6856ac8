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

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// ------------------------------------------------------------------- router
//
// One wave per token.  A logit is computed in the fixed fp32 order that makes
// the selection reproducible: lane l accumulates h[j] * w[j][e] with fma over
// j = l, l+64, ... ascending, then lane partials are added in a halving tree
// that pairs lane l with lane l+s for s = 32, 16, ..., 1 (lane 0 ends with
// the result); a bias is added once afterwards.

constexpr int kRouterWaves = 4;
constexpr int kLogitBlock = 16;  // experts accumulated per pass over h

template <typename W>
__device__ void wave_logits(const W* __restrict__ hrow, const W* __restrict__ wr,
                            const float* __restrict__ bias, int d, int E,
                            float* __restrict__ out /* LDS [E] */) {
  const int lane = threadIdx.x & 63;
  for (int e0 = 0; e0 < E; e0 += kLogitBlock) {
    const int ne = min(kLogitBlock, E - e0);
    float acc[kLogitBlock];
#pragma unroll
    for (int q = 0; q < kLogitBlock; ++q) acc[q] = 0.0f;
    for (int j = lane; j < d; j += 64) {
      const float hj = to_f32(hrow[j]);
      const W* row = wr + static_cast<size_t>(j) * E + e0;
#pragma unroll
      for (int q = 0; q < kLogitBlock; ++q)
        if (q < ne) acc[q] = fmaf(hj, to_f32(row[q]), acc[q]);
    }
#pragma unroll
    for (int q = 0; q < kLogitBlock; ++q) {
      float v = acc[q];
#pragma unroll
      for (int s = 32; s >= 1; s >>= 1) v = v + __shfl_down(v, s, 64);
      if (lane == 0 && q < ne) {
        if (bias != nullptr) v = v + bias[e0 + q];
        out[e0 + q] = v;
      }
    }
  }
}

template <typename W>
__global__ __launch_bounds__(64 * kRouterWaves) void router_kernel(RouterArgs a) {
  extern __shared__ __align__(16) float rl_smem[];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * kRouterWaves + wave;
  const bool active = t < a.T;  // no early return: the block syncs below
  float* logits = rl_smem + wave * a.E;
  const W* hrow = static_cast<const W*>(a.h) + static_cast<size_t>(active ? t : 0) * a.d;

  if (a.wr != nullptr) {
    if (active) wave_logits<W>(hrow, static_cast<const W*>(a.wr), a.bias, a.d, a.E, logits);
    __syncthreads();
    if (active) {
      // K rounds of wave argmax over the untaken experts: the larger logit
      // wins, the lower index on equal logits.
      uint64_t taken = 0;  // bit q: expert lane + 64 q taken (E <= 4096)
      float m = 0.0f, zsel = 0.0f, my_ex = 0.0f;
      int my_idx = 0;
      for (int k = 0; k < a.K; ++k) {
        float bv = -INFINITY;
        int bi = 0x7fffffff;
        for (int q = 0, e = lane; e < a.E; ++q, e += 64) {
          if ((taken >> q) & 1ull) continue;
          float v = logits[e];
          if (v != v) v = -INFINITY;  // NaN ranks last, so an index is always found
          if (v > bv || (v == bv && e < bi)) {
            bv = v;
            bi = e;
          }
        }
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) {
          const float ov = __shfl_xor(bv, s, 64);
          const int oi = __shfl_xor(bi, s, 64);
          if (ov > bv || (ov == bv && oi < bi)) {
            bv = ov;
            bi = oi;
          }
        }
        if ((bi & 63) == lane) taken |= 1ull << (bi >> 6);
        if (k == 0) m = bv;  // the first pick is the largest logit
        const float ex = expf(bv - m);
        zsel += ex;
        if (lane == k) {
          my_ex = ex;
          my_idx = bi;
        }
      }
      float z = zsel;
      if (!a.renormalize) {
        float part = 0.0f;
        for (int e = lane; e < a.E; e += 64) part += expf(logits[e] - m);
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) part += __shfl_xor(part, s, 64);
        z = part;
      }
      if (lane < a.K) {
        a.idx[static_cast<size_t>(t) * a.K + lane] = my_idx;
        a.w[static_cast<size_t>(t) * a.K + lane] = my_ex / z;
      }
    }
    __syncthreads();
  }

  if (a.wr_next != nullptr) {
    if (active) wave_logits<W>(hrow, static_cast<const W*>(a.wr_next), a.bias_next, a.d, a.E, logits);
    __syncthreads();
    if (active) {
      float m = -INFINITY;
      for (int e = lane; e < a.E; e += 64) m = fmaxf(m, logits[e]);
#pragma unroll
      for (int s = 32; s >= 1; s >>= 1) m = fmaxf(m, __shfl_xor(m, s, 64));
      float z = 0.0f;
      for (int e = lane; e < a.E; e += 64) z += expf(logits[e] - m);
#pragma unroll
      for (int s = 32; s >= 1; s >>= 1) z += __shfl_xor(z, s, 64);
      for (int e = lane; e < a.E; e += 64)
        a.p_pred[static_cast<size_t>(t) * a.E + e] = expf(logits[e] - m) / z;
    }
  }
}

hipError_t launch_router(const RouterArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  const dim3 grid((a.T + kRouterWaves - 1) / kRouterWaves);
  const size_t lds = sizeof(float) * kRouterWaves * a.E;
  if (a.dtype == kBF16)
    hipLaunchKernelGGL(router_kernel<uint16_t>, grid, dim3(64 * kRouterWaves), lds, s, a);
  else
    hipLaunchKernelGGL(router_kernel<float>, grid, dim3(64 * kRouterWaves), lds, s, a);
  return hipGetLastError();
}

// ----------------------------------------------------------------- grouping
//
// Stable counting sort of the T*K slots by expert in one work-group:
// histogram, exclusive scan, then blocks of 1024 slots placed in slot order
// (within a wave by ballot rank, across waves by per-wave counts).

constexpr int kGroupThreads = 1024;
constexpr int kGroupWaves = kGroupThreads / 64;

__global__ __launch_bounds__(kGroupThreads) void group_kernel(GroupArgs a) {
  __shared__ int cnt[kMaxExperts];
  __shared__ int base[kMaxExperts];
  __shared__ int wcnt[kGroupWaves][kMaxExperts];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int e = tid; e < a.E; e += kGroupThreads) cnt[e] = 0;
  __syncthreads();
  // indices come from the router kernel and lie in [0, E); the clamp only
  // keeps LDS accesses in bounds whatever the input
  for (int s = tid; s < a.TK; s += kGroupThreads) atomicAdd(&cnt[min(max(a.idx[s], 0), a.E - 1)], 1);
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int e = 0; e < a.E; ++e) {
      base[e] = run;
      a.offsets[e] = run;
      if (a.host_offsets) a.host_offsets[e] = run;
      run += cnt[e];
    }
    a.offsets[a.E] = run;
    if (a.host_offsets) a.host_offsets[a.E] = run;
  }
  __syncthreads();
  const uint64_t lt = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
  for (int b0 = 0; b0 < a.TK; b0 += kGroupThreads) {
    for (int i = tid; i < kGroupWaves * a.E; i += kGroupThreads) (&wcnt[0][0])[(i / a.E) * kMaxExperts + i % a.E] = 0;
    __syncthreads();
    const int s = b0 + tid;
    const int e = (s < a.TK) ? min(max(a.idx[s], 0), a.E - 1) : -1;
    int rank = 0;
    uint64_t pending = __ballot(e >= 0);
    while (pending) {
      const int leader = __ffsll(static_cast<unsigned long long>(pending)) - 1;
      const int le = __shfl(e, leader, 64);
      const uint64_t same = __ballot(e == le);
      if (e == le) rank = __popcll(same & lt);
      if (lane == leader) wcnt[wave][le] = __popcll(same);
      pending &= ~same;
    }
    __syncthreads();
    if (e >= 0) {
      int p = base[e] + rank;
      for (int w2 = 0; w2 < wave; ++w2) p += wcnt[w2][e];
      a.perm[p] = s;
      a.pos[s] = p;
    }
    __syncthreads();
    for (int e2 = tid; e2 < a.E; e2 += kGroupThreads) {
      int add = 0;
      for (int w2 = 0; w2 < kGroupWaves; ++w2) add += wcnt[w2][e2];
      base[e2] += add;
    }
    __syncthreads();
  }
  if (a.host_offsets) __threadfence_system();
}

hipError_t launch_group(const GroupArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(group_kernel, dim3(1), dim3(kGroupThreads), 0, s, a);
  return hipGetLastError();
}

// ------------------------------------------------------ prediction ranking

constexpr int kRankThreads = 1024;

__global__ __launch_bounds__(kRankThreads) void rank_kernel(RankArgs a) {
  __shared__ float part[kRankThreads];
  __shared__ float score[kMaxExperts];
  const int tid = threadIdx.x;
  int epad = 1;
  while (epad < a.E) epad <<= 1;
  const int G = kRankThreads / epad;  // token groups (>= 2 for E <= 512)
  const int e = tid % epad, g = tid / epad;
  float acc = 0.0f;
  if (e < a.E && g < G)
    for (int t = g; t < a.T; t += G) acc += a.p_pred[static_cast<size_t>(t) * a.E + e];
  part[tid] = acc;
  __syncthreads();
  if (tid < a.E) {
    float s = 0.0f;
    for (int g2 = 0; g2 < G; ++g2) s += part[g2 * epad + tid];
    score[tid] = s;
  }
  __syncthreads();
  if (tid < a.E) {
    const float v = score[tid];
    int r = 0;
    for (int o = 0; o < a.E; ++o) {
      const float u = score[o];
      r += (u > v) || (u == v && o < tid);
    }
    a.order[r] = tid;
    a.score[tid] = v;
    if (a.host_order) a.host_order[r] = tid;
    if (a.host_score) a.host_score[tid] = v;
  }
  if (a.host_order) __threadfence_system();
}

hipError_t launch_rank(const RankArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(rank_kernel, dim3(1), dim3(kRankThreads), 0, s, a);
  return hipGetLastError();
}

// --------------------------------------------------------------- SwiGLU FFN
//
// One work-group computes one 64-unit chunk c of one expert for all of the
// expert's tokens, NT tokens at a time:
//   phase 1: a[t][f] = silu(h_t . G_f) * (h_t . U_f) for the chunk's units f
//            (8 waves x 8 units, 8 lanes per unit row, 16-byte loads);
//   phase 2: y[t][:] = sum_f a[t][f] * D_f (each thread owns VEC columns);
//   writes y as the chunk's fp32 partial row of that token.
// Chunk layout (model dtype): [G: 64 x d][U: 64 x d][D: 64 x d], rows
// d-contiguous.  The same code serves resident and streamed chunks.

template <typename W, int NT, int Q>
__global__ __launch_bounds__(kFfnThreads) void ffn_chunk_kernel(FfnArgs a) {
  constexpr int VEC = Vec<W>::N;
  extern __shared__ __align__(16) unsigned char ffn_smem[];
  const int d = a.d;
  const int wg = blockIdx.x;
  int ti = 0;
  for (int i = 1; i < a.n_tasks; ++i)
    if (a.tasks[i].wg_begin <= wg) ti = i;
  const FfnTask tk = a.tasks[ti];
  const int c = tk.chunk_lo + (wg - tk.wg_begin);
  const bool routed = tk.expert >= 0;
  int p0 = 0, n_tok = a.T;
  if (routed) {
    p0 = a.offsets[tk.expert];
    n_tok = a.offsets[tk.expert + 1] - p0;
  }
  if (n_tok <= 0) return;

  const size_t cd = static_cast<size_t>(kChunkUnits) * d;
  const W* G = reinterpret_cast<const W*>(tk.base + static_cast<size_t>(c) * a.chunk_bytes);
  const W* U = G + cd;
  const W* D = U + cd;
  float* part = routed ? a.part : a.part_sh + static_cast<size_t>(-1 - tk.expert) * a.sh_plane;
  const int rows = routed ? a.rows_routed : a.rows_shared;

  W* hs = reinterpret_cast<W*>(ffn_smem);                                  // [NT][d]
  float* as = reinterpret_cast<float*>(ffn_smem + sizeof(W) * NT * d);     // [NT][64]
  const W* hsrc = static_cast<const W*>(a.h);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane & 7, grp = lane >> 3;
  const int unit = wave * 8 + grp;  // 8 waves x 8 units = 64

  for (int tile = 0; tile < n_tok; tile += NT) {
    const int nt = min(NT, n_tok - tile);
    // stage the tile's activations in LDS (zero rows past nt)
    const int vec_per_row = d / VEC;
    for (int i = tid; i < NT * vec_per_row; i += kFfnThreads) {
      const int t = i / vec_per_row, k = (i - t * vec_per_row) * VEC;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (t < nt) {
        const int tok = routed ? a.perm[p0 + tile + t] / a.K : tile + t;
        v = *reinterpret_cast<const uint4*>(hsrc + static_cast<size_t>(tok) * d + k);
      }
      *reinterpret_cast<uint4*>(hs + static_cast<size_t>(t) * d + k) = v;
    }
    __syncthreads();

    // phase 1: gate/up dot products of this wave's 8 units
    {
      float ag[NT], au[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) ag[t] = au[t] = 0.0f;
      const W* grow = G + static_cast<size_t>(unit) * d;
      const W* urow = U + static_cast<size_t>(unit) * d;
#pragma unroll 4
      for (int k0 = sub * VEC; k0 < d; k0 += 8 * VEC) {
        float gv[VEC], uv[VEC];
        load16(grow + k0, gv);
        load16(urow + k0, uv);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          float hv[VEC];
          load16(hs + static_cast<size_t>(t) * d + k0, hv);
#pragma unroll
          for (int i = 0; i < VEC; ++i) {
            ag[t] = fmaf(gv[i], hv[i], ag[t]);
            au[t] = fmaf(uv[i], hv[i], au[t]);
          }
        }
      }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int s = 1; s <= 4; s <<= 1) {
          ag[t] += __shfl_xor(ag[t], s, 64);
          au[t] += __shfl_xor(au[t], s, 64);
        }
      }
      if (sub == 0) {
#pragma unroll
        for (int t = 0; t < NT; ++t) as[t * kChunkUnits + unit] = silu(ag[t]) * au[t];
      }
    }
    __syncthreads();

    // phase 2: partial down-projection of the chunk
    {
      float y[NT][Q][VEC];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int q = 0; q < Q; ++q)
#pragma unroll
          for (int i = 0; i < VEC; ++i) y[t][q][i] = 0.0f;
#pragma unroll 4
      for (int f = 0; f < kChunkUnits; ++f) {
        const W* drow = D + static_cast<size_t>(f) * d;
        float av[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) av[t] = as[t * kChunkUnits + f];
#pragma unroll
        for (int q = 0; q < Q; ++q) {
          const int col = (tid + kFfnThreads * q) * VEC;
          if (col < d) {
            float dv[VEC];
            load16(drow + col, dv);
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
              for (int i = 0; i < VEC; ++i) y[t][q][i] = fmaf(av[t], dv[i], y[t][q][i]);
          }
        }
      }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t < nt) {
          const int row = routed ? (p0 + tile + t) : (tile + t);
          float* dst = part + (static_cast<size_t>(c) * rows + row) * d;
#pragma unroll
          for (int q = 0; q < Q; ++q) {
            const int col = (tid + kFfnThreads * q) * VEC;
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
}

template <typename W, int NT, int Q>
static hipError_t launch_ffn_one(const FfnArgs& a, hipStream_t s) {
  const size_t lds = sizeof(W) * NT * a.d + sizeof(float) * NT * kChunkUnits;
  hipLaunchKernelGGL((ffn_chunk_kernel<W, NT, Q>), dim3(a.n_wg), dim3(kFfnThreads), lds, s, a);
  return hipGetLastError();
}

// Only the (NT, Q) pairs whose accumulators fit (NT * Q * VEC <= 64) exist.
template <typename W>
static hipError_t dispatch_ffn(const FfnArgs& a, int nt, int q, hipStream_t s) {
  constexpr int V = Vec<W>::N;
#define MSK_FFN_CASE(NT_, Q_)                                          \
  if (nt == NT_ && q == Q_) {                                          \
    if constexpr (NT_ * Q_ * V <= 64) return launch_ffn_one<W, NT_, Q_>(a, s); \
  }
  MSK_FFN_CASE(1, 1) MSK_FFN_CASE(2, 1) MSK_FFN_CASE(4, 1) MSK_FFN_CASE(8, 1)
  MSK_FFN_CASE(1, 2) MSK_FFN_CASE(2, 2) MSK_FFN_CASE(4, 2) MSK_FFN_CASE(8, 2)
  MSK_FFN_CASE(1, 4) MSK_FFN_CASE(2, 4) MSK_FFN_CASE(4, 4) MSK_FFN_CASE(8, 4)
#undef MSK_FFN_CASE
  return hipErrorInvalidValue;
}

// Tokens per tile: the smallest of {1, 2, 4, 8} covering max_tok, limited so
// that the LDS tile stays within 64 KiB and the accumulators NT*Q*VEC <= 64.
static int pick_nt(int max_tok, int d, int elem, int q, int vec) {
  int nt = 1;
  while (nt < max_tok && nt < 8) nt <<= 1;
  while (nt > 1 &&
         (static_cast<size_t>(nt) * (static_cast<size_t>(d) * elem + sizeof(float) * kChunkUnits) > 65536 ||
          nt * q * vec > 64))
    nt >>= 1;
  return nt;
}

hipError_t launch_ffn(const FfnArgs& a, int max_tok, hipStream_t s) {
  if (a.n_wg <= 0 || a.n_tasks <= 0) return hipSuccess;
  const int vec = (a.dtype == kBF16) ? 8 : 4;
  const int elem = (a.dtype == kBF16) ? 2 : 4;
  const int q = (a.d + kFfnThreads * vec - 1) / (kFfnThreads * vec);
  const int qq = q <= 1 ? 1 : (q <= 2 ? 2 : 4);
  if (q > 4) return hipErrorInvalidValue;
  const int nt = pick_nt(max_tok, a.d, elem, qq, vec);
  return (a.dtype == kBF16) ? dispatch_ffn<uint16_t>(a, nt, qq, s) : dispatch_ffn<float>(a, nt, qq, s);
}

// ------------------------------------------------------------------ combine
//
// One work-group of 16 waves per (token, 256 columns).  Wave w sums chunks
// c = w, w+16, ... of one (token, k) partial; the 16 wave sums are added in
// wave order; the k terms are added in selection order with their gate
// weights, then the shared experts in index order.  The order is fixed, so
// the output is the same whichever stream or launch produced each chunk.

constexpr int kCombineWaves = 16;

__device__ __forceinline__ float4 f4add(float4 x, float4 y) {
  return make_float4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
}

__global__ __launch_bounds__(64 * kCombineWaves) void combine_kernel(CombineArgs a) {
  __shared__ float4 red[kCombineWaves][64];
  const int t = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.y * 256 + lane * 4;
  const bool live = col < a.d;
  float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
  const int n_terms = a.K + a.n_shared;
  for (int term = 0; term < n_terms; ++term) {
    const bool routed = term < a.K;
    const float* base;
    int row, rows, nch;
    if (routed) {
      base = a.part;
      row = a.pos[t * a.K + term];
      rows = a.rows_routed;
      nch = a.n_chunks;
    } else {
      base = a.part_sh + static_cast<size_t>(term - a.K) * a.sh_plane;
      row = t;
      rows = a.rows_shared;
      nch = a.n_chunks_sh;
    }
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (live)
      for (int c = wave; c < nch; c += kCombineWaves)
        s = f4add(s, *reinterpret_cast<const float4*>(base + (static_cast<size_t>(c) * rows + row) * a.d + col));
    red[wave][lane] = s;
    __syncthreads();
    if (wave == 0) {
      float4 tot = red[0][lane];
      for (int w2 = 1; w2 < kCombineWaves; ++w2) tot = f4add(tot, red[w2][lane]);
      if (routed) {
        const float wk = a.w[t * a.K + term];
        y = make_float4(fmaf(wk, tot.x, y.x), fmaf(wk, tot.y, y.y), fmaf(wk, tot.z, y.z), fmaf(wk, tot.w, y.w));
      } else {
        y = f4add(y, tot);
      }
    }
    __syncthreads();
  }
  if (wave == 0 && live) *reinterpret_cast<float4*>(a.y + static_cast<size_t>(t) * a.d + col) = y;
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  const dim3 grid(a.T, (a.d + 255) / 256);
  hipLaunchKernelGGL(combine_kernel, grid, dim3(64 * kCombineWaves), 0, s, a);
  return hipGetLastError();
}

}  // namespace msk
