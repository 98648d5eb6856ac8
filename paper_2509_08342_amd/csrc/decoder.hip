// Kernels of the decoder loop around the split-expert MoE layer (Sec. 2.1:
// an attention module, Eq. (1), then the MoE module, Eq. (2), per layer;
// the head after the last layer): dense projections, rotary embedding with
// the key/value cache append, causal grouped-query attention, greedy token
// choice and the embedding gather.  Stateless entry points: every buffer is
// the caller's, every call is enqueued on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"
#include "moesplit.h"

namespace {

constexpr int kDenseThreads = 256;
constexpr int kDenseRows = 8;        // output rows per work-group (two per wave)
constexpr int kAttThreads = 256;
constexpr int kAttWideThreads = 1024;  // single-token steps
constexpr int kAttMaxScores = 16000;  // floats of queries and scores a work-group keeps in LDS (< 64 KiB)

__device__ __forceinline__ void bf16x8_to_f32(uint4 v, float (&o)[8]) {
  o[0] = __uint_as_float(v.x << 16);
  o[1] = __uint_as_float(v.x & 0xffff0000u);
  o[2] = __uint_as_float(v.y << 16);
  o[3] = __uint_as_float(v.y & 0xffff0000u);
  o[4] = __uint_as_float(v.z << 16);
  o[5] = __uint_as_float(v.z & 0xffff0000u);
  o[6] = __uint_as_float(v.w << 16);
  o[7] = __uint_as_float(v.w & 0xffff0000u);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// ------------------------------------------------------------------ dense
//
// y[t][o] = sum_i x[t][i] W[o][i] (+ add[t][o]): W [n_out][n_in] bf16 rows
// (the nn.Linear layout), x bf16, y fp32.  A work-group takes 8 output rows,
// two per wave; lanes stride over the row in 16-byte pieces with every
// piece of a row requested before use; NT tokens of x sit in LDS per pass.
template <int NT, int PJ>
__global__ __launch_bounds__(kDenseThreads) void dense_kernel(const uint16_t* __restrict__ x,
                                                              const uint16_t* __restrict__ w,
                                                              const float* __restrict__ add, float* __restrict__ y,
                                                              int T, int n_in, int n_out) {
  extern __shared__ __align__(16) uint16_t xs[];  // [NT][n_in]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row0 = blockIdx.x * kDenseRows + 2 * wave;
  const int pieces = n_in / 8;
  constexpr int PMAX = PJ;  // pieces per lane at the largest n_in of this variant
  for (int t0 = 0; t0 < T; t0 += NT) {
    const int nt = min(NT, T - t0);
    __syncthreads();  // the previous tile's readers are done
    for (int i = tid; i < NT * pieces; i += kDenseThreads) {
      const int t = i / pieces, p = i - t * pieces;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (t < nt) v = *reinterpret_cast<const uint4*>(x + static_cast<size_t>(t0 + t) * n_in + 8 * p);
      *reinterpret_cast<uint4*>(xs + static_cast<size_t>(t) * n_in + 8 * p) = v;
    }
    __syncthreads();
    float acc[2][NT];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[r][t] = 0.0f;
    uint4 wv[2][PMAX];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int row = min(row0 + r, n_out - 1);  // clamped: rows past n_out are not stored
#pragma unroll
      for (int j = 0; j < PMAX; ++j) {
        const int p = lane + 64 * j;
        if (p < pieces) wv[r][j] = *reinterpret_cast<const uint4*>(w + static_cast<size_t>(row) * n_in + 8 * p);
      }
    }
#pragma unroll
    for (int j = 0; j < PMAX; ++j) {
      const int p = lane + 64 * j;
      if (p < pieces) {
        float wf[2][8];
        bf16x8_to_f32(wv[0][j], wf[0]);
        bf16x8_to_f32(wv[1][j], wf[1]);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          float xf[8];
          bf16x8_to_f32(*reinterpret_cast<const uint4*>(xs + static_cast<size_t>(t) * n_in + 8 * p), xf);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            acc[0][t] = fmaf(wf[0][e], xf[e], acc[0][t]);
            acc[1][t] = fmaf(wf[1][e], xf[e], acc[1][t]);
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) acc[r][t] += __shfl_xor(acc[r][t], s, 64);
      }
    if (lane == 0) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int row = row0 + r;
        if (row < n_out) {
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            if (t < nt) {
              const size_t o = static_cast<size_t>(t0 + t) * n_out + row;
              y[o] = acc[r][t] + (add ? add[o] : 0.0f);
            }
          }
        }
      }
    }
  }
}

// ------------------------------------------------------ rotary + KV append
//
// Block (t, head): heads [0, Hq) are query heads (rotated into q_out),
// [Hq, Hq + Hkv) key heads (rotated into the key cache at position
// pos0 + t), [Hq + Hkv, Hq + 2 Hkv) value heads (copied into the value
// cache).  Thread i < D/2 rotates the pair (i, i + D/2) by the angle
// p * base^(-2 i / D), computed in double precision.
__global__ void rope_kv_kernel(const float* __restrict__ qkv, int Hq, int Hkv, int D, int pos0, double log2_base,
                               uint16_t* __restrict__ q_out, uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                               int max_ctx) {
  const int t = blockIdx.x, head = blockIdx.y;
  const int width = (Hq + 2 * Hkv) * D;
  const float* src = qkv + static_cast<size_t>(t) * width + static_cast<size_t>(head) * D;
  const int pos = pos0 + t;
  const int half = D / 2;
  for (int i = threadIdx.x; i < half; i += blockDim.x) {
    const float x1 = src[i], x2 = src[i + half];
    if (head >= Hq + Hkv) {  // value head: stored as is
      uint16_t* dst = vc + (static_cast<size_t>(head - Hq - Hkv) * max_ctx + pos) * D;
      dst[i] = f32_to_bf16(x1);
      dst[i + half] = f32_to_bf16(x2);
      continue;
    }
    const double ang = static_cast<double>(pos) * exp2(-2.0 * i / D * log2_base);
    double sn, cs;
    sincos(ang, &sn, &cs);
    const float c = static_cast<float>(cs), s = static_cast<float>(sn);
    const float r1 = x1 * c - x2 * s, r2 = x2 * c + x1 * s;
    uint16_t* dst = head < Hq ? q_out + (static_cast<size_t>(t) * Hq + head) * D
                              : kc + (static_cast<size_t>(head - Hq) * max_ctx + pos) * D;
    dst[i] = f32_to_bf16(r1);
    dst[i + half] = f32_to_bf16(r2);
  }
}

// ------------------------------------------------------------- attention
//
// Block (t, g): the G = Hq / Hkv query heads of key/value group g for token
// t, over positions 0 .. pos0 + t, in BLK threads (1024 for a single-token
// step, whose T x Hkv blocks alone would leave most of the GPU idle; 256
// otherwise).  Scores in LDS ([G][n]); softmax with the
// row maximum subtracted; then p . V over the positions.
template <int BLK>
__device__ __forceinline__ float block_reduce(float v, bool is_max, float* red) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) {
    const float o = __shfl_xor(v, s, 64);
    v = is_max ? fmaxf(v, o) : v + o;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float r = red[0];
  for (int w = 1; w < BLK / 64; ++w) r = is_max ? fmaxf(r, red[w]) : r + red[w];
  return r;
}

template <int G, int BLK>
__global__ __launch_bounds__(BLK) void attention_kernel(const uint16_t* __restrict__ q,
                                                                const uint16_t* __restrict__ kc,
                                                                const uint16_t* __restrict__ vc, int Hq, int Hkv,
                                                                int D, int pos0, int max_ctx,
                                                                uint16_t* __restrict__ out) {
  extern __shared__ __align__(16) float att_smem[];  // qf [G][D], scores [G][n], wave sums [4][G][D]
  __shared__ float red[BLK / 64];
  const int t = blockIdx.x, g = blockIdx.y, tid = threadIdx.x;
  const int n = pos0 + t + 1;
  float* qf = att_smem;
  float* sc = att_smem + G * D;
  for (int i = tid; i < G * D; i += BLK)
    qf[i] = bf16_to_f32(q[(static_cast<size_t>(t) * Hq + g * G) * D + i]);
  __syncthreads();
  const float scale = 1.0f / sqrtf(static_cast<float>(D));
  const uint16_t* K = kc + static_cast<size_t>(g) * max_ctx * D;
  const uint16_t* V = vc + static_cast<size_t>(g) * max_ctx * D;
  for (int p = tid; p < n; p += BLK) {
    float s[G];
#pragma unroll
    for (int h = 0; h < G; ++h) s[h] = 0.0f;
    for (int k8 = 0; k8 < D; k8 += 8) {
      float kf[8];
      bf16x8_to_f32(*reinterpret_cast<const uint4*>(K + static_cast<size_t>(p) * D + k8), kf);
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) s[h] = fmaf(qf[h * D + k8 + e], kf[e], s[h]);
    }
#pragma unroll
    for (int h = 0; h < G; ++h) sc[h * n + p] = s[h] * scale;
  }
  __syncthreads();
  for (int h = 0; h < G; ++h) {
    float m = -INFINITY;
    for (int p = tid; p < n; p += BLK) m = fmaxf(m, sc[h * n + p]);
    m = block_reduce<BLK>(m, true, red);
    float sum = 0.0f;
    for (int p = tid; p < n; p += BLK) {
      const float e = expf(sc[h * n + p] - m);
      sc[h * n + p] = e;
      sum += e;
    }
    sum = block_reduce<BLK>(sum, false, red);
    __syncthreads();
    for (int p = tid; p < n; p += BLK) sc[h * n + p] /= sum;
  }
  __syncthreads();
  // p . V: thread (position lane pl, column group cg) sums 8 columns of every
  // head over positions pl, pl + PL, ... (one 16-byte V load serves all G
  // heads); the position lanes of a wave are combined with shuffles, the
  // waves' sums through LDS (after the scores, which stay in use until then)
  const int CG = D / 8, PL = BLK / CG;
  const int cg = tid % CG, pl = tid / CG;
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
  if (pl < PL) {
    for (int p = pl; p < n; p += PL) {
      float vf[8];
      bf16x8_to_f32(*reinterpret_cast<const uint4*>(V + static_cast<size_t>(p) * D + 8 * cg), vf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float pr = sc[h * n + p];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pr, vf[e], acc[h][e]);
      }
    }
  }
  // lanes l and l ^ (CG * 2^j) hold the same columns for other positions
  for (int m = CG; m < 64; m <<= 1)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] += __shfl_xor(acc[h][e], m, 64);
  float* wsum = sc + G * n;  // [waves][G][D]
  const int lane = tid & 63, wave = tid >> 6;
  if (lane < CG && CG <= 64) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) wsum[(wave * G + h) * D + 8 * cg + e] = acc[h][e];
  }
  __syncthreads();
  for (int o = tid; o < G * D; o += BLK) {
    float v = 0.0f;
    for (int w = 0; w < BLK / 64; ++w) v += wsum[w * G * D + o];
    const int h = o / D, col = o - h * D;
    out[(static_cast<size_t>(t) * Hq + g * G + h) * D + col] = f32_to_bf16(v);
  }
}

// ---------------------------------------------------------- arg max, gather

__global__ __launch_bounds__(256) void argmax_kernel(const float* __restrict__ x, int n, int32_t* __restrict__ idx) {
  __shared__ float bv[4];
  __shared__ int bi[4];
  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* row = x + static_cast<size_t>(t) * n;
  float v = -INFINITY;
  int i = n;
  for (int j = tid; j < n; j += 256) {
    const float xv = row[j];
    if (xv > v) {  // ascending j per thread: the first maximum stays
      v = xv;
      i = j;
    }
  }
  for (int s = 32; s >= 1; s >>= 1) {
    const float ov = __shfl_xor(v, s, 64);
    const int oi = __shfl_xor(i, s, 64);
    if (ov > v || (ov == v && oi < i)) {
      v = ov;
      i = oi;
    }
  }
  if (lane == 0) {
    bv[wave] = v;
    bi[wave] = i;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < 4; ++w)
      if (bv[w] > v || (bv[w] == v && bi[w] < i)) {
        v = bv[w];
        i = bi[w];
      }
    idx[t] = i < n ? i : 0;
  }
}

__global__ void embed_kernel(const int32_t* __restrict__ ids, const uint16_t* __restrict__ table, int n_vocab,
                             int d, uint16_t* __restrict__ out) {
  const int t = blockIdx.x;
  const int id = min(max(ids[t], 0), n_vocab - 1);  // ids are validated by the argmax; clamped to stay in bounds
  const uint4* src = reinterpret_cast<const uint4*>(table + static_cast<size_t>(id) * d);
  uint4* dst = reinterpret_cast<uint4*>(out + static_cast<size_t>(t) * d);
  for (int i = threadIdx.x; i < d / 8; i += blockDim.x) dst[i] = src[i];
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Prompts (T >= kDenseMmaTokens, n_in a multiple of 32): the same product on
// the matrix cores, v_mfma_f32_16x16x32_bf16 (lane l holds A[row l % 16][8 k
// from 8 (l / 16)], B[8 k from 8 (l / 16)][column l % 16] and C[rows
// 4 (l / 16) + r][column l % 16]).  A work-group takes 64 tokens x 64
// outputs, wave w the outputs 16 w .. 16 w + 15 of all four 16-token blocks.
// x [T][n_in] and W [n_out][n_in] are both contiguous along k, so each
// fragment is one 16-byte load; loads run kDenseKb k steps of 32 ahead.
// Tokens past T and outputs past n_out are clamped on load, never stored.
constexpr int kDenseMmaTokens = 16;
constexpr int kDenseKb = 2;

typedef __bf16 dbf16x8_t __attribute__((ext_vector_type(8)));
typedef float df32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ df32x4_t dmfma(uint4 a, uint4 b, df32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(dbf16x8_t, a), __builtin_bit_cast(dbf16x8_t, b),
                                                 c, 0, 0, 0);
}

__global__ __launch_bounds__(256) void dense_mma_kernel(const uint16_t* __restrict__ x,
                                                        const uint16_t* __restrict__ w,
                                                        const float* __restrict__ add, float* __restrict__ y, int T,
                                                        int n_in, int n_out) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int t0 = blockIdx.x * 64, o0 = blockIdx.y * 64 + 16 * wave;
  const int n = lane & 15, kq = 8 * (lane >> 4);
  const uint16_t* wrow = w + static_cast<size_t>(min(o0 + n, n_out - 1)) * n_in + kq;
  const uint16_t* xrow[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) xrow[rb] = x + static_cast<size_t>(min(t0 + 16 * rb + n, T - 1)) * n_in + kq;
  const int ksteps = n_in / 32;
  df32x4_t acc[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) acc[rb] = df32x4_t{0.f, 0.f, 0.f, 0.f};
  uint4 bn[kDenseKb], an[kDenseKb][4], bc[kDenseKb], ac[kDenseKb][4];
  auto load = [&](int s0) {
#pragma unroll
    for (int u = 0; u < kDenseKb; ++u) {
      const int k = min(s0 + u, ksteps - 1) * 32;  // clamped past the last step; used only in range
      bn[u] = *reinterpret_cast<const uint4*>(wrow + k);
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) an[u][rb] = *reinterpret_cast<const uint4*>(xrow[rb] + k);
    }
  };
  load(0);
  for (int s0 = 0; s0 < ksteps; s0 += kDenseKb) {
#pragma unroll
    for (int u = 0; u < kDenseKb; ++u) {
      bc[u] = bn[u];
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) ac[u][rb] = an[u][rb];
    }
    load(s0 + kDenseKb);
#pragma unroll
    for (int u = 0; u < kDenseKb; ++u)
      if (s0 + u < ksteps) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) acc[rb] = dmfma(ac[u][rb], bc[u], acc[rb]);
      }
  }
  const int o = o0 + n;
  if (o < n_out) {
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = t0 + 16 * rb + 4 * (lane >> 4) + r;
        if (t < T) {
          const size_t i = static_cast<size_t>(t) * n_out + o;
          y[i] = acc[rb][r] + (add ? add[i] : 0.0f);
        }
      }
  }
}

ms_status launched() { return hipGetLastError() == hipSuccess ? MS_OK : MS_E_HIP; }

}  // namespace

extern "C" {

ms_status ms_dense(const void* x, const void* w, int32_t T, int32_t n_in, int32_t n_out, float* y, const float* add,
                   void* stream) {
  if (T < 0 || n_in <= 0 || n_out <= 0) return MS_E_INVALID;
  if (T == 0) return MS_OK;
  if (!x || !w || !y || !aligned16(x) || !aligned16(w)) return MS_E_INVALID;
  if (n_in % 8 != 0 || n_in > 8192) return MS_E_UNSUPPORTED;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid((n_out + kDenseRows - 1) / kDenseRows);
  const auto* xp = static_cast<const uint16_t*>(x);
  const auto* wp = static_cast<const uint16_t*>(w);
  if (T >= kDenseMmaTokens && n_in % 32 == 0) {
    hipLaunchKernelGGL(dense_mma_kernel, dim3((T + 63) / 64, (n_out + 63) / 64), dim3(256), msk::kGuardLds, s, xp, wp,
                       add, y, T, n_in, n_out);
    return launched();
  }
  if (n_in <= 4096)
    hipLaunchKernelGGL((dense_kernel<4, 8>), grid, dim3(kDenseThreads), 4 * n_in * 2, s, xp, wp, add, y, T, n_in,
                       n_out);
  else
    hipLaunchKernelGGL((dense_kernel<2, 16>), grid, dim3(kDenseThreads), 2 * n_in * 2, s, xp, wp, add, y, T, n_in,
                       n_out);
  return launched();
}

ms_status ms_rope_kv(const float* qkv, int32_t T, int32_t Hq, int32_t Hkv, int32_t D, int32_t pos0, double base,
                     void* q_out, void* k_cache, void* v_cache, int32_t max_ctx, void* stream) {
  if (T < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || pos0 < 0 || max_ctx <= 0 || !(base > 1.0)) return MS_E_INVALID;
  if (T == 0) return MS_OK;
  if (!qkv || !q_out || !k_cache || !v_cache) return MS_E_INVALID;
  if (D % 2 != 0 || Hq % Hkv != 0) return MS_E_INVALID;
  if (static_cast<int64_t>(pos0) + T > max_ctx) return MS_E_INVALID;
  hipLaunchKernelGGL(rope_kv_kernel, dim3(T, Hq + 2 * Hkv), dim3(64), msk::kGuardLds, static_cast<hipStream_t>(stream), qkv, Hq,
                     Hkv, D, pos0, log2(base), static_cast<uint16_t*>(q_out), static_cast<uint16_t*>(k_cache),
                     static_cast<uint16_t*>(v_cache), max_ctx);
  return launched();
}

ms_status ms_attention(const void* q, const void* k_cache, const void* v_cache, int32_t T, int32_t Hq, int32_t Hkv,
                       int32_t D, int32_t pos0, int32_t max_ctx, void* out, void* stream) {
  if (T < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || pos0 < 0 || max_ctx <= 0) return MS_E_INVALID;
  if (T == 0) return MS_OK;
  if (!q || !k_cache || !v_cache || !out || !aligned16(k_cache) || !aligned16(v_cache)) return MS_E_INVALID;
  if (Hq % Hkv != 0 || static_cast<int64_t>(pos0) + T > max_ctx) return MS_E_INVALID;
  const int G = Hq / Hkv;
  if (D < 8 || D > 512 || (D & (D - 1)) != 0 || G > 8 || static_cast<int64_t>(G) * (5 * D + pos0 + T) > kAttMaxScores)
    return MS_E_UNSUPPORTED;
  // LDS: queries [G][D], scores [G][n], per-wave p.V sums [waves][G][D]
  const bool wide = T == 1 && static_cast<int64_t>(G) * ((1 + kAttWideThreads / 64) * D + pos0 + T) <= kAttMaxScores;
  const int waves = (wide ? kAttWideThreads : kAttThreads) / 64;
  const size_t lds = sizeof(float) * static_cast<size_t>(G) * ((1 + waves) * D + pos0 + T);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const auto* qp = static_cast<const uint16_t*>(q);
  const auto* kp = static_cast<const uint16_t*>(k_cache);
  const auto* vp = static_cast<const uint16_t*>(v_cache);
  auto* op = static_cast<uint16_t*>(out);
  const dim3 grid(T, Hkv);
#define MSK_ATT_CASE(G_)                                                                                   \
  case G_:                                                                                                 \
    if (wide)                                                                                              \
      hipLaunchKernelGGL((attention_kernel<G_, kAttWideThreads>), grid, dim3(kAttWideThreads), lds, s, qp, kp, vp, \
                         Hq, Hkv, D, pos0, max_ctx, op);                                                   \
    else                                                                                                   \
      hipLaunchKernelGGL((attention_kernel<G_, kAttThreads>), grid, dim3(kAttThreads), lds, s, qp, kp, vp, Hq, \
                         Hkv, D, pos0, max_ctx, op);                                                       \
    break;
  switch (G) {
    MSK_ATT_CASE(1)
    MSK_ATT_CASE(2)
    MSK_ATT_CASE(4)
    MSK_ATT_CASE(8)
    default: return MS_E_UNSUPPORTED;
  }
#undef MSK_ATT_CASE
  return launched();
}

ms_status ms_argmax(const float* x, int32_t T, int32_t n, int32_t* idx_out, void* stream) {
  if (T < 0 || n <= 0) return MS_E_INVALID;
  if (T == 0) return MS_OK;
  if (!x || !idx_out) return MS_E_INVALID;
  hipLaunchKernelGGL(argmax_kernel, dim3(T), dim3(256), 0, static_cast<hipStream_t>(stream), x, n, idx_out);
  return launched();
}

ms_status ms_embed(const int32_t* ids, const void* table, int32_t n_vocab, int32_t T, int32_t d, void* out,
                   void* stream) {
  if (T < 0 || n_vocab <= 0 || d <= 0) return MS_E_INVALID;
  if (T == 0) return MS_OK;
  if (!ids || !table || !out || !aligned16(table) || !aligned16(out) || d % 8 != 0) return MS_E_INVALID;
  hipLaunchKernelGGL(embed_kernel, dim3(T), dim3(256), msk::kGuardLds, static_cast<hipStream_t>(stream), ids,
                     static_cast<const uint16_t*>(table), n_vocab, d, static_cast<uint16_t*>(out));
  return launched();
}

}  // extern "C"
