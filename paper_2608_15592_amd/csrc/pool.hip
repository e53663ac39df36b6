// Fusion and pooling, Eq. 3 - Eq. 5 (Section 4.2):
//   T_i = lambda1 S_i + lambda2 H_i,  e_i = softmax_{prompt}(T_i / alpha),  h_b = sum_i e_i x_i
//
// The weights are never normalised before pooling.  pool_partial_kernel
// (workgroup = 256-token chunk x prompt x 2048-feature slice) forms
// u_i = T_i / alpha for its rows, the chunk's own max m_c (and first arg-max),
// p_i = exp(u_i - m_c) and exp-sum s_c with wave reductions only, and streams
// X once: each thread owns 8 consecutive hidden features (one 16-byte bf16
// load per row, 8 rows in flight) and accumulates sum_i p_i x_i in fp32.
// pool_finish_kernel combines the chunks of each prompt in a fixed order,
// weighting chunk c by exp(m_c - M) / Z (M the prompt max, Z its exp-sum),
// which is exactly sum_i e_i x_i; it also writes the arg-max token and, when
// asked, the normalised weights e.  With z-scored or min-max scaled inputs a
// per-prompt statistics pass (zscore_stats_kernel, minmax_stats_kernel) runs
// first and gives u = c1 (S - centre_S) + c2 (H - centre_H).  Batches of
// (nearly) equal-length prompts that fill the chip by themselves take one kernel
// instead (pool_prompt_kernel: a workgroup streams a whole prompt for one
// feature slice, so there are no chunk partials to combine), and so do other
// batches of prompts up to 8192 tokens (pool_ragged_kernel: the slice width
// follows each prompt's length); the chunked pair serves longer prompts.  No
// atomics: results are bitwise reproducible.
#include <algorithm>

#include "estp_common.h"

namespace estp {
namespace detail {

constexpr int kThreads = 256;
constexpr int kChunk = 256;                // rows per pooling workgroup (= threads of the weights kernel)
constexpr int kSlice = kThreads * 8;       // hidden features per pooling workgroup
constexpr float kZEps = 1e-6f;
constexpr int kMaxChunks = 1024;           // chunks per prompt the finisher stages (prompts up to 256k tokens)
constexpr int kFinishBatch = 8;            // chunk partials the finisher loads at once

struct ChunkStat {
  float m;    // max of u over the chunk
  float s;    // sum of 2^((u - m) log2 e) over the chunk
  int idx;    // lowest row (prompt-local) attaining m
  int pad;
};

__device__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  float r = 0.f;
  const int nw = blockDim.x >> 6;
  for (int i = 0; i < nw; ++i) r += sh[i];
  return r;
}

// (max value, lowest index attaining it) over the workgroup
__device__ void block_argmax(float& v, int& idx, float* shv, int* shi) {
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(v, o, 64);
    const int oi = __shfl_xor(idx, o, 64);
    if (ov > v || (ov == v && oi < idx)) {
      v = ov;
      idx = oi;
    }
  }
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) {
    shv[w] = v;
    shi[w] = idx;
  }
  __syncthreads();
  v = shv[0];
  idx = shi[0];
  const int nw = blockDim.x >> 6;
  for (int i = 1; i < nw; ++i)
    if (shv[i] > v || (shv[i] == v && shi[i] < idx)) {
      v = shv[i];
      idx = shi[i];
    }
}

__device__ double block_sum_d(double v, double* sh) {
  v = wave_sum_d(v);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  double r = 0.0;
  const int nw = blockDim.x >> 6;
  for (int i = 0; i < nw; ++i) r += sh[i];
  return r;
}

// Per-prompt coefficients (c1, c2, centre_S, centre_H) of u = c1 (S - centre_S) + c2 (H - centre_H)
// for z-scored inputs: (lambda1 (S - mean_S) / (std_S + eps) + lambda2 (H - mean_H) / (std_H + eps))
// / alpha.  Mean and variance are taken in fp64, and the centre stays a separate term: when a
// prompt's values are nearly equal, S - centre is then (nearly) exact and the fp32 rounding of the
// centre shifts every u of the prompt alike, which the softmax ignores.  (Folding it into one
// constant would cancel two large terms for std ~ 0.)
__global__ __launch_bounds__(1024) void zscore_stats_kernel(const float* __restrict__ S, const float* __restrict__ H,
                                                            const int* __restrict__ cu, float a1, float a2,
                                                            float4* __restrict__ coef) {
  __shared__ double sh[16];
  const int b = blockIdx.x;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  double ss = 0.0, sv = 0.0;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    ss += double(S[base + i]);
    sv += double(H[base + i]);
  }
  const double ms = block_sum_d(ss, sh) / N;
  const double mh = block_sum_d(sv, sh) / N;
  double vs = 0.0, vh = 0.0;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    const double ds = double(S[base + i]) - ms, dh = double(H[base + i]) - mh;
    vs += ds * ds;
    vh += dh * dh;
  }
  const double sds = sqrt(block_sum_d(vs, sh) / N);
  const double sdh = sqrt(block_sum_d(vh, sh) / N);
  if (threadIdx.x == 0) {
    const double c1 = double(a1) / (sds + double(kZEps)), c2 = double(a2) / (sdh + double(kZEps));
    coef[b] = make_float4(float(c1), float(c2), float(ms), float(mh));
  }
}

__device__ float block_reduce_max(float v, float* sh) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  float r = -INFINITY;
  const int nw = blockDim.x >> 6;
  for (int i = 0; i < nw; ++i) r = fmaxf(r, sh[i]);
  return r;
}

// Per-prompt coefficients (c1, c2, min_S, min_H) of u = c1 (S - min_S) + c2 (H - min_H) for min-max
// scaled inputs: (lambda1 (S - min_S) / (max_S - min_S + eps) + lambda2 (H - min_H) / (max_H - min_H
// + eps)) / alpha.
__global__ __launch_bounds__(1024) void minmax_stats_kernel(const float* __restrict__ S, const float* __restrict__ H,
                                                            const int* __restrict__ cu, float a1, float a2,
                                                            float4* __restrict__ coef) {
  __shared__ float sh[16];
  const int b = blockIdx.x;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  float xs = -INFINITY, ns = -INFINITY, xh = -INFINITY, nh = -INFINITY;  // max and -min
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    const float sv = S[base + i], hv = H[base + i];
    xs = fmaxf(xs, sv);
    ns = fmaxf(ns, -sv);
    xh = fmaxf(xh, hv);
    nh = fmaxf(nh, -hv);
  }
  xs = block_reduce_max(xs, sh);
  ns = block_reduce_max(ns, sh);
  xh = block_reduce_max(xh, sh);
  nh = block_reduce_max(nh, sh);
  if (threadIdx.x == 0) {
    const float c1 = a1 / ((xs + ns) + kZEps), c2 = a2 / ((xh + nh) + kZEps);
    coef[b] = make_float4(c1, c2, -ns, -nh);
  }
}

// One row's 8 consecutive features as loaded (raw), and their fp32 values.
template <typename T>
struct Row8;
template <>
struct Row8<uint16_t> {  // 8 bf16 in one 16-byte load
  using Raw = uint4;
  __device__ static __forceinline__ Raw load(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ static __forceinline__ void fma8(float w, const Raw& q, float (&acc)[8]) {
    const uint32_t x[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[2 * k] = fmaf(w, __uint_as_float(x[k] << 16), acc[2 * k]);
      acc[2 * k + 1] = fmaf(w, __uint_as_float(x[k] & 0xffff0000u), acc[2 * k + 1]);
    }
  }
};
template <>
struct Row8<float> {  // 8 fp32 in two 16-byte loads
  struct Raw {
    float4 a, b;
  };
  __device__ static __forceinline__ Raw load(const float* p) {
    return Raw{*reinterpret_cast<const float4*>(p), *reinterpret_cast<const float4*>(p + 4)};
  }
  __device__ static __forceinline__ void fma8(float w, const Raw& q, float (&acc)[8]) {
    acc[0] = fmaf(w, q.a.x, acc[0]); acc[1] = fmaf(w, q.a.y, acc[1]);
    acc[2] = fmaf(w, q.a.z, acc[2]); acc[3] = fmaf(w, q.a.w, acc[3]);
    acc[4] = fmaf(w, q.b.x, acc[4]); acc[5] = fmaf(w, q.b.y, acc[5]);
    acc[6] = fmaf(w, q.b.z, acc[6]); acc[7] = fmaf(w, q.b.w, acc[7]);
  }
};

__device__ __forceinline__ float4 coef_of(const float4* coef, int b, float a1, float a2) {
  return coef ? coef[b] : make_float4(a1, a2, 0.f, 0.f);
}

// u = c1 (S - centre_S) + c2 (H - centre_H) for coefficients (c1, c2, centre_S, centre_H)
__device__ __forceinline__ float fused_score(const float4& cf, float s, float h) {
  return fmaf(cf.x, s - cf.z, cf.y * (h - cf.w));
}

// Streams one chunk of X.  Every wave forms the chunk's weights by itself
// (wave reductions only, no workgroup barrier), so the first rows of X, which
// do not depend on the weights, are already in flight while they are formed.
template <typename T>
__global__ __launch_bounds__(kThreads) void pool_partial_kernel(const T* __restrict__ X, const float* __restrict__ S,
                                                                const float* __restrict__ H,
                                                                const int* __restrict__ cu, int d, int n_chunk_max,
                                                                float a1, float a2, const float4* __restrict__ coef,
                                                                float* __restrict__ part,
                                                                ChunkStat* __restrict__ cstat, int nslices,
                                                                const int2* __restrict__ chunk_map) {
  __shared__ float wts[kThreads / 64][kChunk];  // one private copy of the chunk weights per wave
  // One workgroup per (chunk, feature slice), slice fastest: the slices of a
  // chunk (the two halves of its 8 KB rows at d = 4096) run together.  The
  // chunk is (prompt, chunk) = (k / n_chunk_max, k % n_chunk_max), or, when
  // many prompts are much shorter than the longest, the k-th entry of the
  // list of live chunks (a grid sized by the longest prompt would be mostly
  // workgroups that exit at once, and those cost ~25 ns each).
  const int slice = blockIdx.x % nslices;
  const int k = blockIdx.x / nslices;
  int b, chunk;
  if (chunk_map) {
    const int2 bc = chunk_map[k];
    if (bc.x < 0) return;  // past the live chunks
    b = bc.x;
    chunk = bc.y;
  } else {
    b = k / n_chunk_max;
    chunk = k % n_chunk_max;
  }
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const int r0 = chunk * kChunk;
  if (r0 >= N) return;
  const int nr = min(N - r0, kChunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = (slice * kThreads + threadIdx.x) * 8;
  const bool active = c < d;
  const T* xp = X + size_t(base + r0) * d + (active ? c : 0);

  constexpr int kInFlight = 8;
  typename Row8<T>::Raw v[kInFlight];
  const int n_first = min(nr, kInFlight);
  if (active) {
#pragma unroll
    for (int k = 0; k < kInFlight; ++k)
      if (k < n_first) v[k] = Row8<T>::load(xp + size_t(k) * d);
  }

  // u for rows lane, lane + 64, ...; wave-wide max (first arg-max), weights, sum
  const float4 cf = coef_of(coef, b, a1, a2);
  constexpr int kPer = kChunk / 64;
  float u[kPer];
  float m = -INFINITY;
  int mi = 0x7fffffff;
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int r = q * 64 + lane;
    u[q] = -INFINITY;
    if (r < nr) {
      const int i = base + r0 + r;
      u[q] = fused_score(cf, S[i], H[i]);
      if (u[q] > m) {  // rows visited in increasing order: strict keeps the first
        m = u[q];
        mi = r0 + r;
      }
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(m, o, 64);
    const int oi = __shfl_xor(mi, o, 64);
    if (om > m || (om == m && oi < mi)) {
      m = om;
      mi = oi;
    }
  }
  float sc = 0.f;
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const float p = fast_exp2((u[q] - m) * kLog2e);  // 0 for rows past the chunk (u = -inf)
    wts[wave][q * 64 + lane] = p;
    sc += p;
  }
  sc = wave_sum(sc);
  if (threadIdx.x == 0 && slice == 0) cstat[size_t(b) * n_chunk_max + chunk] = ChunkStat{m, sc, mi, 0};

  if (!active) return;
  const float* w = wts[wave];
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < kInFlight; ++k)
    if (k < n_first) Row8<T>::fma8(w[k], v[k], acc);
  int r = n_first;
  for (; r + kInFlight <= nr; r += kInFlight) {
#pragma unroll
    for (int k = 0; k < kInFlight; ++k) v[k] = Row8<T>::load(xp + size_t(r + k) * d);
#pragma unroll
    for (int k = 0; k < kInFlight; ++k) Row8<T>::fma8(w[r + k], v[k], acc);
  }
  for (; r < nr; ++r) Row8<T>::fma8(w[r], Row8<T>::load(xp + size_t(r) * d), acc);
  float* out = part + (size_t(b) * n_chunk_max + chunk) * d + c;
  *reinterpret_cast<float4*>(out) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  *reinterpret_cast<float4*>(out + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
}

// One-kernel pooling of whole prompts: workgroup = (prompt, 512-feature slice),
// slice fastest.  All 8 waves form the prompt's weights together (u into LDS,
// workgroup max with its first arg-max, exp-sum Z) while the first rows of X
// are already in flight; wave w then streams rows w, w + 8, ... of the slice
// (one 16-byte load per lane and row, 8 rows in flight), reading its weights as
// LDS broadcasts, and the 8 wave sums are added in wave order and scaled by
// 1/Z.  No chunk partials, no second kernel.  Used for batches of equal-length
// prompts that fill the chip by themselves (the host decides).
constexpr int kPromptThreads = 512;
constexpr int kPromptWaves = kPromptThreads / 64;
constexpr int kPromptSlice = 512;     // hidden features per workgroup: 8 per lane
constexpr int kPromptMaxRows = 8192;  // weights of the prompt staged in LDS (32 KB)

template <typename T>
__global__ __launch_bounds__(kPromptThreads) void pool_prompt_kernel(
    const T* __restrict__ X, const float* __restrict__ S, const float* __restrict__ H, const int* __restrict__ cu,
    int d, int nslices, float a1, float a2, const float4* __restrict__ coef, float* __restrict__ pooled,
    float* __restrict__ e, int* __restrict__ top) {
  __shared__ float wts[kPromptMaxRows];
  __shared__ __attribute__((aligned(16))) float red[kPromptWaves][kPromptSlice];
  __shared__ float shv[kPromptWaves];
  __shared__ int shi[kPromptWaves];
  const int slice = blockIdx.x % nslices;
  const int b = blockIdx.x / nslices;
  const int base = cu[b];
  const int N = min(cu[b + 1] - base, kPromptMaxRows);  // the host guarantees N <= kPromptMaxRows
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = slice * kPromptSlice + lane * 8;
  const bool active = c < d;
  const T* xp = X + size_t(base) * d + (active ? c : 0);
  // rows of this wave: wave, wave + 8, ...
  const int nw = N > wave ? (N - wave + kPromptWaves - 1) / kPromptWaves : 0;

  constexpr int kInFlight = 8;
  typename Row8<T>::Raw v[kInFlight];
  const int n_first = min(nw, kInFlight);
  if (active) {
#pragma unroll
    for (int k = 0; k < kInFlight; ++k)
      if (k < n_first) v[k] = Row8<T>::load(xp + size_t(wave + kPromptWaves * k) * d);
  }

  // u = c1 (S - centre_S) + c2 (H - centre_H) for every token of the prompt, the first arg-max, the exp-sum
  const float4 cf = coef_of(coef, b, a1, a2);
  float m = -INFINITY;
  int mi = 0x7fffffff;
  for (int i = tid; i < N; i += kPromptThreads) {
    const float u = fused_score(cf, S[base + i], H[base + i]);
    wts[i] = u;
    if (u > m) {  // increasing i: strict keeps the first
      m = u;
      mi = i;
    }
  }
  block_argmax(m, mi, shv, shi);
  float z = 0.f;
  for (int i = tid; i < N; i += kPromptThreads) {
    const float p = fast_exp2((wts[i] - m) * kLog2e);
    wts[i] = p;
    z += p;
  }
  z = block_sum(z, shv);  // its barriers also publish wts
  const float invZ = 1.f / z;
  if (slice == 0) {
    if (e)
      for (int i = tid; i < N; i += kPromptThreads) e[base + i] = wts[i] * invZ;
    if (top && tid == 0) top[b] = base + mi;
  }

  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (active) {
    const float* w = wts + wave;  // weight of the wave's q-th row: w[kPromptWaves * q]
#pragma unroll
    for (int k = 0; k < kInFlight; ++k)
      if (k < n_first) Row8<T>::fma8(w[kPromptWaves * k], v[k], acc);
    int q = n_first;
    for (; q + kInFlight <= nw; q += kInFlight) {
#pragma unroll
      for (int k = 0; k < kInFlight; ++k) v[k] = Row8<T>::load(xp + size_t(wave + kPromptWaves * (q + k)) * d);
#pragma unroll
      for (int k = 0; k < kInFlight; ++k) Row8<T>::fma8(w[kPromptWaves * (q + k)], v[k], acc);
    }
    for (; q < nw; ++q) Row8<T>::fma8(w[kPromptWaves * q], Row8<T>::load(xp + size_t(wave + kPromptWaves * q) * d), acc);
  }
  float* rw = &red[wave][lane * 8];
  *reinterpret_cast<float4*>(rw) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  *reinterpret_cast<float4*>(rw + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
  __syncthreads();
  const int f = slice * kPromptSlice + tid;
  if (f < d) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kPromptWaves; ++w) s += red[w][tid];
    pooled[size_t(b) * d + f] = s * invZ;
  }
}

// One-kernel pooling of a ragged batch.  Work unit = (prompt, feature slice),
// like pool_prompt_kernel, but the slice width follows the prompt's length so
// that every unit streams about the same number of bytes of X (512 KB, less
// for small batches: four units per compute unit): a short prompt takes whole
// rows, a 4096-token one 128 of 4096 features.  Each unit sums all rows of its
// prompt for its slice, so there are no partials and no second kernel.  The
// units of a prompt are consecutive; a workgroup finds its (prompt, slice) by
// scanning the prompt lengths itself (no list kernel).  G = F / 8 lanes cover
// one row (16-byte loads), 512 / G rows are in flight per load round and 8
// rounds per thread; the row groups' sums are added in a fixed order.
// Unit size, slice alignment and the narrowest slice were swept on MI355X over
// the ragged, Qwen-shaped and 1B-shaped batches: 512 KB units, widths a
// multiple of 64 features (whole 128-byte lines of bf16), at least 128 features.
constexpr int kRaggedThreads = 512;
constexpr int kRaggedMaxPrompts = 8192;  // prompts the in-kernel scan covers (16 per thread)
constexpr int kRaggedMinSlice = 128;     // narrowest slice (features)
constexpr int kRaggedUnitsPerCu = 4;
constexpr size_t kRaggedMaxUnitBytes = size_t(512) << 10;
constexpr size_t kRaggedMinUnitBytes = size_t(64) << 10;
constexpr int kRaggedAlign = 64;         // slice widths are multiples of this many features

// Width of one of ns slices of d features, a multiple of kRaggedAlign (at least the 8 of a
// 16-byte bf16 load), and never more than the workgroup covers.
__host__ __device__ __forceinline__ int ragged_width(int d, int ns) {
  const int w = ((d + ns - 1) / ns + kRaggedAlign - 1) / kRaggedAlign * kRaggedAlign;
  return w < kRaggedThreads * 8 ? w : ((d + ns - 1) / ns + 7) / 8 * 8;
}

// Fewest slices whose width fits the workgroup (512 lanes x 8 features).
__host__ __device__ __forceinline__ int ragged_min_slices(int d) {
  int ns = 1;
  while (ragged_width(d, ns) > kRaggedThreads * 8) ns *= 2;
  return ns;
}

// Slice width for a prompt of n rows: d split into about (its X bytes) / unit_bytes slices, at
// least ragged_min_slices(d), none narrower than kRaggedMinSlice features.
__host__ __device__ __forceinline__ int ragged_slice_width(int n, int d, int elem_bytes, size_t unit_bytes) {
  const size_t bytes = size_t(n) * size_t(d) * size_t(elem_bytes);
  const size_t lo = size_t(ragged_min_slices(d)), hi = std::max(lo, size_t(d / kRaggedMinSlice));
  return ragged_width(d, int(std::min(hi, std::max(lo, bytes / unit_bytes))));
}

// Units (nonempty slices) of a prompt of n rows.
__host__ __device__ __forceinline__ int ragged_slices(int n, int d, int elem_bytes, size_t unit_bytes) {
  const int w = ragged_slice_width(n, d, elem_bytes, unit_bytes);
  return (d + w - 1) / w;
}

template <typename T>
__global__ __launch_bounds__(kRaggedThreads) void pool_ragged_kernel(
    const T* __restrict__ X, const float* __restrict__ S, const float* __restrict__ H, const int* __restrict__ cu,
    int B, int d, size_t unit_bytes, float a1, float a2, const float4* __restrict__ coef,
    float* __restrict__ pooled, float* __restrict__ e, int* __restrict__ top) {
  __shared__ float wts[kPromptMaxRows];
  __shared__ __attribute__((aligned(16))) float red[kRaggedThreads * 8];
  __shared__ int scan[kRaggedThreads / 64];
  __shared__ int unit[2];
  __shared__ float shv[kRaggedThreads / 64];
  __shared__ int shi[kRaggedThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // ---- which (prompt, slice) is unit blockIdx.x: scan of the per-prompt slice counts
  {
    const int per = (B + kRaggedThreads - 1) / kRaggedThreads;  // <= 16
    const int b0 = min(B, tid * per), b1 = min(B, b0 + per);
    int cnt = 0;
    for (int b = b0; b < b1; ++b) cnt += ragged_slices(cu[b + 1] - cu[b], d, int(sizeof(T)), unit_bytes);
    int x = cnt;  // inclusive scan within the wave, then over the wave totals
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) scan[wave] = x;
    if (tid == 0) unit[0] = -1;
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += scan[w];
    const int k = int(blockIdx.x);
    int first = before + x - cnt;  // this thread's first unit
    if (k >= first && k < first + cnt) {
      for (int b = b0; b < b1; ++b) {
        const int ns = ragged_slices(cu[b + 1] - cu[b], d, int(sizeof(T)), unit_bytes);
        if (k < first + ns) {
          unit[0] = b;
          unit[1] = k - first;
          break;
        }
        first += ns;
      }
    }
    __syncthreads();
  }
  const int b = unit[0];
  if (b < 0) return;  // past the last unit
  const int slice = unit[1];
  const int base = cu[b];
  const int N = min(cu[b + 1] - base, kPromptMaxRows);  // the host guarantees N <= kPromptMaxRows
  const int F = ragged_slice_width(N, d, int(sizeof(T)), unit_bytes);
  const int f0 = slice * F;
  const int G = F / 8;                             // lanes per row
  const int RP = kRaggedThreads / G;              // row groups (F <= 512 x 8: RP >= 1)
  const int col = tid % G, rgrp = tid / G;         // this thread's 8 features and first row
  const int c = f0 + col * 8;
  const bool active = rgrp < RP && c < d;
  const T* xp = X + size_t(base) * d + (active ? c : 0);
  const int nr = active && N > rgrp ? (N - rgrp + RP - 1) / RP : 0;  // rows of this thread: rgrp + RP q

  constexpr int kInFlight = 8;
  typename Row8<T>::Raw v[kInFlight];
  const int n_first = min(nr, kInFlight);
#pragma unroll
  for (int q = 0; q < kInFlight; ++q)
    if (q < n_first) v[q] = Row8<T>::load(xp + size_t(rgrp + RP * q) * d);

  // ---- the prompt's weights: u into LDS, first arg-max, exp-sum
  const float4 cf = coef_of(coef, b, a1, a2);
  float m = -INFINITY;
  int mi = 0x7fffffff;
  for (int i = tid; i < N; i += kRaggedThreads) {
    const float u = fused_score(cf, S[base + i], H[base + i]);
    wts[i] = u;
    if (u > m) {  // increasing i: strict keeps the first
      m = u;
      mi = i;
    }
  }
  block_argmax(m, mi, shv, shi);
  float z = 0.f;
  for (int i = tid; i < N; i += kRaggedThreads) {
    const float p = fast_exp2((wts[i] - m) * kLog2e);
    wts[i] = p;
    z += p;
  }
  z = block_sum(z, shv);  // its barriers also publish wts
  const float invZ = 1.f / z;
  if (slice == 0) {
    if (e)
      for (int i = tid; i < N; i += kRaggedThreads) e[base + i] = wts[i] * invZ;
    if (top && tid == 0) top[b] = base + mi;
  }

  // ---- stream the slice: 8 rows in flight per thread
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const float* w = wts + rgrp;  // weight of this thread's q-th row: w[RP * q]
#pragma unroll
  for (int q = 0; q < kInFlight; ++q)
    if (q < n_first) Row8<T>::fma8(w[RP * q], v[q], acc);
  int q = n_first;
  for (; q + kInFlight <= nr; q += kInFlight) {
#pragma unroll
    for (int k = 0; k < kInFlight; ++k) v[k] = Row8<T>::load(xp + size_t(rgrp + RP * (q + k)) * d);
#pragma unroll
    for (int k = 0; k < kInFlight; ++k) Row8<T>::fma8(w[RP * (q + k)], v[k], acc);
  }
  for (; q < nr; ++q) Row8<T>::fma8(w[RP * q], Row8<T>::load(xp + size_t(rgrp + RP * q) * d), acc);

  // ---- add the RP row groups of each feature in a fixed order
  float* rw = red + tid * 8;
  *reinterpret_cast<float4*>(rw) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  *reinterpret_cast<float4*>(rw + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
  __syncthreads();
  for (int f = tid; f < F; f += kRaggedThreads) {
    if (f0 + f >= d) break;
    float sum = 0.f;
    for (int g = 0; g < RP; ++g) sum += red[(g * G + f / 8) * 8 + f % 8];
    pooled[size_t(b) * d + f0 + f] = sum * invZ;
  }
}

// List of live chunks: entry k = (prompt, chunk) in prompt order, then
// (-1, 0) up to n_bound.  One workgroup: each thread counts the chunks of a
// run of consecutive prompts, an exclusive scan over the threads places them.
// Counts are capped at n_chunk_max and writes at n_bound, so a max_seqlen below
// the longest prompt (invalid input) stays inside the workspace.
__global__ __launch_bounds__(1024) void chunk_map_kernel(const int* __restrict__ cu, int B, int n_chunk_max,
                                                         int n_bound, int2* __restrict__ map) {
  __shared__ int wsum[16];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int per = (B + 1023) / 1024;
  const int b0 = min(B, t * per), b1 = min(B, b0 + per);
  int cnt = 0;
  for (int b = b0; b < b1; ++b) cnt += min((cu[b + 1] - cu[b] + kChunk - 1) / kChunk, n_chunk_max);
  // inclusive scan within the wave, then over the 16 wave totals
  int x = cnt;
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int before = 0, total = 0;
  for (int i = 0; i < 16; ++i) {
    before += (i < w) ? wsum[i] : 0;
    total += wsum[i];
  }
  int k = before + x - cnt;  // exclusive prefix: this thread's first entry
  for (int b = b0; b < b1; ++b) {
    const int nc = min((cu[b + 1] - cu[b] + kChunk - 1) / kChunk, n_chunk_max);
    for (int c = 0; c < nc && k < n_bound; ++c) map[k++] = make_int2(b, c);
  }
  for (int i = total + t; i < n_bound; i += 1024) map[i] = make_int2(-1, 0);
}

// Combine the chunks of prompt b in a fixed order:
// pooled = sum_c 2^((m_c - M) log2 e) partial_c / Z,  Z = sum_c 2^((m_c - M) log2 e) s_c.
// Workgroups x < nslices each finish a 2048-feature slice; the rest write the
// normalised weights e of kThreads tokens each (when asked); x = 0 writes the
// top token.  Every load that does not need the chunk statistics (the token's
// S and H, the first kFinishBatch chunk partials) is issued before them, so the
// kernel costs about two memory round trips.
__global__ __launch_bounds__(kThreads) void pool_finish_kernel(const float* __restrict__ part,
                                                               const ChunkStat* __restrict__ cstat,
                                                               const float* __restrict__ S,
                                                               const float* __restrict__ H,
                                                               const int* __restrict__ cu, int d, int n_chunk_max,
                                                               int nslices, int n_finish, float a1, float a2,
                                                               const float4* __restrict__ coef,
                                                               float* __restrict__ pooled, float* __restrict__ e,
                                                               int* __restrict__ top) {
  __shared__ ChunkStat cs[kMaxChunks];
  const int slice = blockIdx.x % n_finish;  // n_finish workgroups per prompt
  const int b = blockIdx.x / n_finish;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const int nch = min((N + kChunk - 1) / kChunk, n_chunk_max);
  const bool weights = slice >= nslices;
  if (weights && !e) return;
  const int wi = (slice - nslices) * kThreads + threadIdx.x;  // weights slice: this thread's token
  float sv = 0.f, hv = 0.f;
  if (weights && wi < N) {
    sv = S[base + wi];
    hv = H[base + wi];
  }
  const int c = (slice * kThreads + threadIdx.x) * 8;  // pooling slice: this thread's 8 features
  const bool pool = !weights && c < d;
  const float* p = part + size_t(b) * n_chunk_max * d + c;
  float4 x[2 * kFinishBatch];
  auto load_batch = [&](int k) {
#pragma unroll
    for (int j = 0; j < kFinishBatch; ++j) {
      if (k + j < nch) {
        x[2 * j] = *reinterpret_cast<const float4*>(p + size_t(k + j) * d);
        x[2 * j + 1] = *reinterpret_cast<const float4*>(p + size_t(k + j) * d + 4);
      }
    }
  };
  if (pool) load_batch(0);

  for (int k = threadIdx.x; k < nch; k += kThreads) cs[k] = cstat[size_t(b) * n_chunk_max + k];
  __syncthreads();
  float M = -INFINITY;
  int Mi = 0;
  for (int k = 0; k < nch; ++k)
    if (cs[k].m > M) {  // strict: the first chunk attaining the max keeps the lowest index
      M = cs[k].m;
      Mi = cs[k].idx;
    }
  float Z = 0.f;
  for (int k = 0; k < nch; ++k) Z += cs[k].s * fast_exp2((cs[k].m - M) * kLog2e);
  const float invZ = 1.f / Z;

  if (weights) {
    if (wi < N) {
      const float4 cf = coef_of(coef, b, a1, a2);
      const float u = fused_score(cf, sv, hv);
      e[base + wi] = fast_exp2((u - M) * kLog2e) * invZ;
    }
    return;
  }
  if (slice == 0 && top && threadIdx.x == 0) top[b] = base + Mi;
  if (pool) {
    // chunks summed in ascending order, kFinishBatch partials in flight at a time
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int k = 0; k < nch; k += kFinishBatch) {
      if (k > 0) load_batch(k);
#pragma unroll
      for (int j = 0; j < kFinishBatch; ++j) {
        if (k + j < nch) {
          const float w = fast_exp2((cs[k + j].m - M) * kLog2e) * invZ;
          acc[0] = fmaf(w, x[2 * j].x, acc[0]);
          acc[1] = fmaf(w, x[2 * j].y, acc[1]);
          acc[2] = fmaf(w, x[2 * j].z, acc[2]);
          acc[3] = fmaf(w, x[2 * j].w, acc[3]);
          acc[4] = fmaf(w, x[2 * j + 1].x, acc[4]);
          acc[5] = fmaf(w, x[2 * j + 1].y, acc[5]);
          acc[6] = fmaf(w, x[2 * j + 1].z, acc[6]);
          acc[7] = fmaf(w, x[2 * j + 1].w, acc[7]);
        }
      }
    }
    float* out = pooled + size_t(b) * d + c;
    *reinterpret_cast<float4*>(out) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    *reinterpret_cast<float4*>(out + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
}

}  // namespace detail
}  // namespace estp

using namespace estp;
using namespace estp::detail;

namespace {
// Upper bound on the chunks that hold tokens: sum_b ceil(N_b / kChunk) <= n_tok / kChunk + B.
size_t live_chunk_bound(int64_t n_tok, int32_t B, int32_t max_seqlen) {
  const size_t nch = (size_t(max_seqlen) + kChunk - 1) / kChunk;
  return std::min(size_t(B) * nch, size_t(n_tok) / kChunk + size_t(B));
}

// The one-kernel path streams a whole prompt per workgroup, so it needs prompts of
// (nearly) equal length, short enough for their weights to fit in LDS, and enough
// (prompt, slice) workgroups to fill every compute unit in equal rounds.
bool use_prompt_path(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t d) {
  if (max_seqlen > kPromptMaxRows) return false;
  if (size_t(B) * size_t(max_seqlen) * 8 > size_t(n_tok) * 9) return false;  // > 12.5% below the longest
  const int n_cu = current_device_cu_count();
  if (n_cu < 1) return false;
  const size_t wg = size_t(B) * ((size_t(d) + kPromptSlice - 1) / kPromptSlice);
  return wg >= size_t(n_cu) && (wg % size_t(n_cu) == 0 || wg >= 4 * size_t(n_cu));
}
// Prompts no longer than the LDS weight buffer, and few enough for the in-kernel scan: one kernel
// with length-sized feature slices (pool_ragged_kernel) instead of chunk partials and a finisher.
bool use_ragged_path(int32_t B, int32_t max_seqlen) {
  return max_seqlen <= kPromptMaxRows && B <= kRaggedMaxPrompts;
}

// X bytes per unit: about four units per compute unit over the batch, within [64 KB, 512 KB].
size_t ragged_unit_bytes(int64_t n_tok, int32_t d, size_t esz) {
  const int n_cu = std::max(1, current_device_cu_count());
  const size_t total = size_t(n_tok) * size_t(d) * esz;
  return std::min(kRaggedMaxUnitBytes, std::max(kRaggedMinUnitBytes, total / (size_t(kRaggedUnitsPerCu) * size_t(n_cu))));
}

// Upper bound on sum_b ragged_slices(N_b): a prompt of bytes_b takes at most
// max(min slices, bytes_b / unit) slices (the nonempty ones of that width are no more), so the sum
// is at most total / unit + B * min slices; never more than d / kRaggedMinSlice (or the minimum)
// per prompt.
size_t ragged_unit_bound(int64_t n_tok, int32_t B, int32_t d, size_t esz, size_t unit) {
  const size_t per_max = std::max<size_t>(size_t(ragged_min_slices(d)), size_t(d) / kRaggedMinSlice);
  const size_t bound = size_t(n_tok) * size_t(d) * esz / unit + size_t(B) * size_t(ragged_min_slices(d));
  return std::min(bound, size_t(B) * per_max);
}
}  // namespace

extern "C" size_t estp_combine_pool_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t d,
                                                   int dtype) {
  (void)dtype;
  if (n_tok < 1 || B < 1 || max_seqlen < 1 || d < 1) return 0;
  const size_t nch = (size_t(max_seqlen) + kChunk - 1) / kChunk;
  Carver c(nullptr);
  c.take<float4>(size_t(B));            // per-prompt coefficients (z-score)
  c.take<ChunkStat>(size_t(B) * nch);   // chunk statistics
  c.take<float>(size_t(B) * nch * d);   // chunk partials
  c.take<int2>(live_chunk_bound(n_tok, B, max_seqlen));  // list of live chunks
  return c.bytes();
}

extern "C" int estp_combine_pool(const void* X, const float* S, const float* H, const int32_t* cu_seqlens, int32_t B,
                                 int32_t max_seqlen, int64_t n_tok, int32_t d, float lambda1, float lambda2,
                                 float alpha, int norm, int dtype, float* pooled, float* e, int32_t* top,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  ESTP_REQUIRE(X && S && H && cu_seqlens && pooled, ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: X, S, H, cu_seqlens and pooled must be non-null");
  ESTP_REQUIRE(B >= 1 && max_seqlen >= 1, ESTP_ERR_INVALID_ARG, "estp_combine_pool: B and max_seqlen must be >= 1");
  ESTP_REQUIRE(n_tok >= 1 && n_tok <= INT32_MAX && max_seqlen <= n_tok, ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: n_tok must be in [max_seqlen, 2^31)");
  ESTP_REQUIRE(d >= 8 && d % 8 == 0, ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: d must be a positive multiple of 8, got %d", d);
  ESTP_REQUIRE(alpha > 0.f && alpha < INFINITY, ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: alpha must be finite and > 0");
  ESTP_REQUIRE(lambda1 == lambda1 && lambda2 == lambda2 && fabsf(lambda1) < INFINITY && fabsf(lambda2) < INFINITY,
               ESTP_ERR_INVALID_ARG, "estp_combine_pool: lambda1 and lambda2 must be finite");
  ESTP_REQUIRE(norm == ESTP_NORM_NONE || norm == ESTP_NORM_ZSCORE || norm == ESTP_NORM_MINMAX, ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: unknown norm %d", norm);
  ESTP_REQUIRE(dtype == ESTP_BF16 || dtype == ESTP_F32, ESTP_ERR_INVALID_ARG, "estp_combine_pool: unknown dtype %d",
               dtype);
  ESTP_REQUIRE(aligned(X, 16) && aligned(pooled, 16), ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: X and pooled must be 16-byte aligned");
  ESTP_REQUIRE(max_seqlen <= kMaxChunks * kChunk, ESTP_ERR_UNSUPPORTED,
               "estp_combine_pool: prompts longer than %d tokens are not supported", kMaxChunks * kChunk);
  const size_t need = estp_combine_pool_workspace_size(n_tok, B, max_seqlen, d, dtype);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_combine_pool: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: workspace must be non-null and 256-byte aligned");

  const int nch = (max_seqlen + kChunk - 1) / kChunk;
  const int nslices = (d + kSlice - 1) / kSlice;
  // the full (prompt, chunk) grid, or the list of live chunks when that is clearly shorter
  const size_t n_bound = live_chunk_bound(n_tok, B, max_seqlen);
  const bool use_map = n_bound * 4 < size_t(B) * nch * 3;
  const size_t n_k = use_map ? n_bound : size_t(B) * nch;
  const int ne = e ? (max_seqlen + kThreads - 1) / kThreads : 0;
  const int n_finish = nslices + ne;
  ESTP_REQUIRE(fits_launch(n_k * nslices, kThreads) && fits_launch(size_t(n_finish) * B, kThreads) &&
                   fits_launch(size_t(B) * ((size_t(d) + kPromptSlice - 1) / kPromptSlice), kPromptThreads) &&
                   fits_launch(size_t(B), 1024),
               ESTP_ERR_UNSUPPORTED, "estp_combine_pool: batch too large for one launch");
  Carver c(workspace);
  float4* coef = c.take<float4>(size_t(B));
  ChunkStat* cstat = c.take<ChunkStat>(size_t(B) * nch);
  float* part = c.take<float>(size_t(B) * nch * d);
  int2* map = c.take<int2>(n_bound);
  const float a1 = lambda1 / alpha, a2 = lambda2 / alpha;
  const float4* cf = nullptr;
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<int> cu_h;  // debug checks: cu_seqlens on the host, checked before any kernel reads it
  if (debug_checks_enabled()) {
    const int st = debug_check_cu("estp_combine_pool", cu_seqlens, B, n_tok, max_seqlen, s, &cu_h);
    if (st != ESTP_OK) return st;
  }
  if (norm == ESTP_NORM_ZSCORE) {
    zscore_stats_kernel<<<dim3(B), dim3(1024), 0, s>>>(S, H, cu_seqlens, a1, a2, coef);
    ESTP_CHECK_LAUNCH("zscore_stats_kernel");
    cf = coef;
  } else if (norm == ESTP_NORM_MINMAX) {
    minmax_stats_kernel<<<dim3(B), dim3(1024), 0, s>>>(S, H, cu_seqlens, a1, a2, coef);
    ESTP_CHECK_LAUNCH("minmax_stats_kernel");
    cf = coef;
  }
  if (use_prompt_path(n_tok, B, max_seqlen, d)) {
    const int ns = (d + kPromptSlice - 1) / kPromptSlice;
    const dim3 pgrid(unsigned(size_t(B) * ns));
    if (dtype == ESTP_BF16) {
      pool_prompt_kernel<uint16_t><<<pgrid, dim3(kPromptThreads), 0, s>>>(
          static_cast<const uint16_t*>(X), S, H, cu_seqlens, int(d), ns, a1, a2, cf, pooled, e, top);
    } else {
      pool_prompt_kernel<float><<<pgrid, dim3(kPromptThreads), 0, s>>>(static_cast<const float*>(X), S, H, cu_seqlens,
                                                                       int(d), ns, a1, a2, cf, pooled, e, top);
    }
    ESTP_CHECK_LAUNCH("pool_prompt_kernel");
    return ESTP_OK;
  }
  if (use_ragged_path(B, max_seqlen)) {
    const size_t esz = dtype == ESTP_BF16 ? 2 : 4;
    const size_t ub = ragged_unit_bytes(n_tok, d, esz);
    const size_t n_units = ragged_unit_bound(n_tok, B, d, esz, ub);
    ESTP_REQUIRE(fits_launch(n_units, kRaggedThreads), ESTP_ERR_UNSUPPORTED,
                 "estp_combine_pool: batch too large for one launch");
    if (dtype == ESTP_BF16) {
      pool_ragged_kernel<uint16_t><<<dim3(unsigned(n_units)), dim3(kRaggedThreads), 0, s>>>(
          static_cast<const uint16_t*>(X), S, H, cu_seqlens, B, int(d), ub, a1, a2, cf, pooled, e, top);
    } else {
      pool_ragged_kernel<float><<<dim3(unsigned(n_units)), dim3(kRaggedThreads), 0, s>>>(
          static_cast<const float*>(X), S, H, cu_seqlens, B, int(d), ub, a1, a2, cf, pooled, e, top);
    }
    ESTP_CHECK_LAUNCH("pool_ragged_kernel");
    return ESTP_OK;
  }
  if (use_map) {
    chunk_map_kernel<<<dim3(1), dim3(1024), 0, s>>>(cu_seqlens, B, nch, int(n_bound), map);
    ESTP_CHECK_LAUNCH("chunk_map_kernel");
    if (debug_checks_enabled()) {  // its definition: (prompt, chunk) in prompt order, then (-1, 0)
      std::vector<int2> expect;
      for (int b = 0; b < B; ++b)
        for (int c = 0; c * kChunk < cu_h[b + 1] - cu_h[b]; ++c) expect.push_back(make_int2(b, c));
      expect.resize(std::max(expect.size(), n_bound), make_int2(-1, 0));
      expect.resize(n_bound);
      const int st = debug_check_list("estp_combine_pool", map, expect, s);
      if (st != ESTP_OK) return st;
    }
  }
  const dim3 grid(unsigned(n_k * nslices));
  const int2* cmap = use_map ? map : nullptr;
  if (dtype == ESTP_BF16) {
    pool_partial_kernel<uint16_t><<<grid, dim3(kThreads), 0, s>>>(static_cast<const uint16_t*>(X), S, H, cu_seqlens,
                                                                  int(d), nch, a1, a2, cf, part, cstat, nslices, cmap);
  } else {
    pool_partial_kernel<float><<<grid, dim3(kThreads), 0, s>>>(static_cast<const float*>(X), S, H, cu_seqlens, int(d),
                                                               nch, a1, a2, cf, part, cstat, nslices, cmap);
  }
  ESTP_CHECK_LAUNCH("pool_partial_kernel");
  pool_finish_kernel<<<dim3(unsigned(size_t(n_finish) * B)), dim3(kThreads), 0, s>>>(
      part, cstat, S, H, cu_seqlens, int(d), nch, nslices, n_finish, a1, a2, cf, pooled, e, top);
  ESTP_CHECK_LAUNCH("pool_finish_kernel");
  return ESTP_OK;
}
