// Fusion and pooling, Eq. 3 - Eq. 5 (Section 4.2):
//   T_i = lambda1 S_i + lambda2 H_i,  e_i = softmax_{prompt}(T_i / alpha),  h_b = sum_i e_i x_i
//
// combine_kernel: one workgroup per prompt computes the (optional) z-scores,
// the max and exp-sum of T / alpha, writes e and the argmax token.  Traffic is
// ~16 bytes per token.
//
// pool_partial_kernel: the bandwidth-bound part.  Workgroup (chunk, prompt,
// d-slice) streams kChunk rows of X: each thread owns 8 consecutive hidden
// features (one 16-byte load of bf16 per row), accumulates e_i * x_i in fp32
// with 8 rows in flight, and writes one fp32 partial row.  pool_reduce_kernel
// sums the chunk partials of each prompt in a fixed order (deterministic, no
// atomics).
#include "estp_common.h"

namespace estp {
namespace detail {

constexpr int kCombineThreads = 1024;
constexpr int kPoolThreads = 256;
constexpr int kChunk = 256;                     // rows per pooling workgroup
constexpr int kSlice = kPoolThreads * 8;        // hidden features per pooling workgroup
constexpr float kZEps = 1e-6f;

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

// (max value, lowest index attaining it)
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

__global__ __launch_bounds__(kCombineThreads) void combine_kernel(const float* __restrict__ S,
                                                                  const float* __restrict__ H,
                                                                  const int* __restrict__ cu, float lambda1,
                                                                  float lambda2, float inv_alpha, int zscore,
                                                                  float* __restrict__ e, float* __restrict__ stats,
                                                                  int* __restrict__ top) {
  __shared__ float shv[kCombineThreads / 64];
  __shared__ int shi[kCombineThreads / 64];
  const int b = blockIdx.x;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const float* s = S + base;
  const float* h = H + base;

  // effective coefficients: T/alpha = a1 * S + a2 * H + const (const drops out of the softmax)
  float a1 = lambda1 * inv_alpha, a2 = lambda2 * inv_alpha, c0 = 0.f;
  if (zscore) {
    float ss = 0.f, sh = 0.f;
    for (int i = threadIdx.x; i < N; i += blockDim.x) {
      ss += s[i];
      sh += h[i];
    }
    const float ms = block_sum(ss, shv) / N;
    const float mh = block_sum(sh, shv) / N;
    float vs = 0.f, vh = 0.f;
    for (int i = threadIdx.x; i < N; i += blockDim.x) {
      vs += (s[i] - ms) * (s[i] - ms);
      vh += (h[i] - mh) * (h[i] - mh);
    }
    const float sds = sqrtf(block_sum(vs, shv) / N);
    const float sdh = sqrtf(block_sum(vh, shv) / N);
    a1 /= (sds + kZEps);
    a2 /= (sdh + kZEps);
    c0 = -(a1 * ms + a2 * mh);
  }
  // u_i = T_i / alpha; max with lowest index
  float mx = -INFINITY;
  int mi = 0x7fffffff;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    const float u = fmaf(a1, s[i], fmaf(a2, h[i], c0));
    if (u > mx) {
      mx = u;
      mi = i;
    }
  }
  block_argmax(mx, mi, shv, shi);
  float z = 0.f;
  for (int i = threadIdx.x; i < N; i += blockDim.x)
    z += fast_exp2((fmaf(a1, s[i], fmaf(a2, h[i], c0)) - mx) * kLog2e);
  const float Z = block_sum(z, shv);
  const float invZ = 1.f / Z;
  for (int i = threadIdx.x; i < N; i += blockDim.x)
    e[base + i] = fast_exp2((fmaf(a1, s[i], fmaf(a2, h[i], c0)) - mx) * kLog2e) * invZ;
  if (threadIdx.x == 0) {
    if (top) top[b] = base + mi;
    if (stats) {
      stats[2 * b] = mx;
      stats[2 * b + 1] = Z;
    }
  }
}

template <typename T>
struct Row8;
template <>
struct Row8<uint16_t> {  // 8 bf16 in one 16-byte load
  __device__ static __forceinline__ void load(const uint16_t* p, float (&v)[8]) {
    const uint4 q = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[2 * k] = __uint_as_float(w[k] << 16);
      v[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
    }
  }
};
template <>
struct Row8<float> {  // 8 fp32 in two 16-byte loads
  __device__ static __forceinline__ void load(const float* p, float (&v)[8]) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
};

template <typename T>
__global__ __launch_bounds__(kPoolThreads) void pool_partial_kernel(const T* __restrict__ X,
                                                                    const float* __restrict__ e,
                                                                    const int* __restrict__ cu, int d,
                                                                    int n_chunk_max, float* __restrict__ part) {
  const int chunk = blockIdx.x;
  const int b = blockIdx.y;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const int r0 = chunk * kChunk;
  if (r0 >= N) return;
  const int r1 = min(N, r0 + kChunk);
  const int c = (blockIdx.z * kPoolThreads + threadIdx.x) * 8;
  if (c >= d) return;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const T* xp = X + size_t(base) * d + c;
  const float* ep = e + base;
  int r = r0;
  for (; r + 8 <= r1; r += 8) {
    float v[8][8];
#pragma unroll
    for (int k = 0; k < 8; ++k) Row8<T>::load(xp + size_t(r + k) * d, v[k]);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float w = ep[r + k];
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] = fmaf(w, v[k][q], acc[q]);
    }
  }
  for (; r < r1; ++r) {
    float v[8];
    Row8<T>::load(xp + size_t(r) * d, v);
    const float w = ep[r];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = fmaf(w, v[q], acc[q]);
  }
  float* out = part + (size_t(b) * n_chunk_max + chunk) * d + c;
  *reinterpret_cast<float4*>(out) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  *reinterpret_cast<float4*>(out + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
}

__global__ __launch_bounds__(256) void pool_reduce_kernel(const float* __restrict__ part, const int* __restrict__ cu,
                                                          int d, int n_chunk_max, float* __restrict__ pooled) {
  const int b = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= d) return;
  const int N = cu[b + 1] - cu[b];
  const int nch = (N + kChunk - 1) / kChunk;
  const float* p = part + size_t(b) * n_chunk_max * d + c;
  float v = 0.f;
  for (int k = 0; k < nch; ++k) v += p[size_t(k) * d];
  pooled[size_t(b) * d + c] = v;
}

}  // namespace detail
}  // namespace estp

using namespace estp;
using namespace estp::detail;

extern "C" size_t estp_combine_pool_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t d,
                                                   int dtype) {
  (void)dtype;
  if (n_tok < 1 || B < 1 || max_seqlen < 1 || d < 1) return 0;
  const size_t nch = (size_t(max_seqlen) + kChunk - 1) / kChunk;
  Carver c(nullptr);
  c.take<float>(size_t(n_tok));          // e (when the caller passes none)
  c.take<float>(size_t(B) * 2);          // per-prompt (max, sum)
  c.take<float>(size_t(B) * nch * d);    // chunk partials
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
  ESTP_REQUIRE(norm == ESTP_NORM_NONE || norm == ESTP_NORM_ZSCORE, ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: unknown norm %d", norm);
  ESTP_REQUIRE(dtype == ESTP_BF16 || dtype == ESTP_F32, ESTP_ERR_INVALID_ARG, "estp_combine_pool: unknown dtype %d",
               dtype);
  ESTP_REQUIRE(aligned(X, 16) && aligned(pooled, 16), ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: X and pooled must be 16-byte aligned");
  const size_t need = estp_combine_pool_workspace_size(n_tok, B, max_seqlen, d, dtype);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_combine_pool: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_combine_pool: workspace must be non-null and 256-byte aligned");

  const int nch = (max_seqlen + kChunk - 1) / kChunk;
  Carver c(workspace);
  float* ews = c.take<float>(size_t(n_tok));
  float* stats = c.take<float>(size_t(B) * 2);
  float* part = c.take<float>(size_t(B) * nch * d);
  float* ew = e ? e : ews;
  hipStream_t s = static_cast<hipStream_t>(stream);

  combine_kernel<<<dim3(B), dim3(kCombineThreads), 0, s>>>(S, H, cu_seqlens, lambda1, lambda2, 1.f / alpha, norm == ESTP_NORM_ZSCORE ? 1 : 0, ew, stats, top);
  ESTP_CHECK_LAUNCH("combine_kernel");
  const dim3 grid(nch, B, (d + kSlice - 1) / kSlice);
  if (dtype == ESTP_BF16) {
    pool_partial_kernel<uint16_t><<<grid, dim3(kPoolThreads), 0, s>>>(static_cast<const uint16_t*>(X), ew, cu_seqlens, int(d), nch, part);
  } else {
    pool_partial_kernel<float><<<grid, dim3(kPoolThreads), 0, s>>>(static_cast<const float*>(X), ew, cu_seqlens, int(d), nch, part);
  }
  ESTP_CHECK_LAUNCH("pool_partial_kernel");
  pool_reduce_kernel<<<dim3((d + 255) / 256, B), dim3(256), 0, s>>>(part, cu_seqlens, int(d), nch, pooled);
  ESTP_CHECK_LAUNCH("pool_reduce_kernel");
  return ESTP_OK;
}
