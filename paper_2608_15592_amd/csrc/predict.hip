// Length head (Section 4.3) and shortest-job-first order (Section 5.4).
//
//   a = act(W1 h + b1)            mlp_partial_kernel (split-K fp32 tiles) + mlp_finish_kernel
//   o = W2 a + b2                 head_out_kernel: one workgroup per prompt
//   K == 1: yhat = o_0;  K > 1: p = softmax(o), yhat = sum_k p_k c_k (Eq. 7), bin = argmax p
//   order: stable ascending argsort of yhat (rank counting, exact and deterministic)
#include "estp_common.h"

namespace estp {
namespace detail {

constexpr int kTB = 32;     // prompts per tile
constexpr int kTH = 32;     // hidden units per tile
constexpr int kTK = 32;     // reduction depth per LDS stage
constexpr int kKChunk = 256;  // reduction range of one split-K workgroup

__device__ __forceinline__ float act_fn(float x, int act) {
  if (act == ESTP_ACT_RELU) return fmaxf(x, 0.f);
  // tanh-form GELU: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))
  const float u = 0.7978845608028654f * fmaf(0.044715f * x, x * x, x);
  return 0.5f * x * (1.f + tanhf(u));
}

// Split-K partial of the first layer: part[z, b, j] = sum_{k in chunk z} P[b, k] W1[j, k].
// 256 threads own a 32 x 32 (prompt x hidden) tile, 4 outputs each; the grid spans
// hidden tiles x prompt tiles x reduction chunks so that W1 is streamed once by
// hundreds of workgroups even for small batches.
__global__ __launch_bounds__(256) void mlp_partial_kernel(const float* __restrict__ P, const float* __restrict__ W1,
                                                          int B, int d, int Hd, float* __restrict__ part) {
  __shared__ float sp[kTK][kTB + 1];
  __shared__ float sw[kTK][kTH + 1];
  const int th = blockIdx.x * kTH, tb = blockIdx.y * kTB, z = blockIdx.z;
  const int k_lo = z * kKChunk, k_hi = min(d, k_lo + kKChunk);
  const int tx = threadIdx.x & 31;         // hidden unit in the tile
  const int ty = (threadIdx.x >> 5) * 4;   // first of 4 prompts
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = k_lo; k0 < k_hi; k0 += kTK) {
    for (int e = threadIdx.x; e < kTB * kTK; e += 256) {
      const int r = e / kTK, k = e % kTK;  // consecutive threads read consecutive k of one row
      const int gk = k0 + k;
      sp[k][r] = (tb + r < B && gk < k_hi) ? P[size_t(tb + r) * d + gk] : 0.f;
      sw[k][r] = (th + r < Hd && gk < k_hi) ? W1[size_t(th + r) * d + gk] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < kTK; ++k) {
      const float w = sw[k][tx];
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] = fmaf(sp[k][ty + i], w, acc[i]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int b = tb + ty + i, j = th + tx;
    if (b < B && j < Hd) part[(size_t(z) * B + b) * Hd + j] = acc[i];
  }
}

// A[b, j] = act(sum_z part[z, b, j] + b1[j]), chunks summed in order.
__global__ __launch_bounds__(256) void mlp_finish_kernel(const float* __restrict__ part, const float* __restrict__ b1,
                                                         int B, int Hd, int nz, int act, float* __restrict__ A) {
  const size_t e = size_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= size_t(B) * Hd) return;
  const int j = int(e % Hd);
  float v = 0.f;
  for (int z = 0; z < nz; ++z) v += part[size_t(z) * B * Hd + e];
  A[e] = act_fn(v + (b1 ? b1[j] : 0.f), act);
}

// One workgroup (256 threads) per prompt: o = W2 a + b2, then y-hat and bin.
__global__ __launch_bounds__(256) void head_out_kernel(const float* __restrict__ A, const float* __restrict__ W2,
                                                       const float* __restrict__ b2, const float* __restrict__ centres,
                                                       int Hd, int K, float* __restrict__ o_ws,
                                                       float* __restrict__ yhat, int* __restrict__ bin) {
  __shared__ float red[4];
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* a = A + size_t(b) * Hd;
  float* o = o_ws + size_t(b) * K;
  for (int k = wave; k < K; k += 4) {  // one wave per output, lanes over the hidden units
    const float* w = W2 + size_t(k) * Hd;
    float v = 0.f;
    for (int j = lane; j < Hd; j += 64) v = fmaf(w[j], a[j], v);
    v = wave_sum(v);
    if (lane == 0) o[k] = v + (b2 ? b2[k] : 0.f);
  }
  __syncthreads();
  if (K == 1) {
    if (threadIdx.x == 0) yhat[b] = o[0];
    return;
  }
  if (wave != 0) return;
  // softmax over K bins, expectation over the centres, argmax (lowest index)
  float mx = -INFINITY;
  int mi = 0x7fffffff;
  for (int k = lane; k < K; k += 64)
    if (o[k] > mx) {
      mx = o[k];
      mi = k;
    }
  for (int off = 32; off > 0; off >>= 1) {
    const float ov = __shfl_xor(mx, off, 64);
    const int oi = __shfl_xor(mi, off, 64);
    if (ov > mx || (ov == mx && oi < mi)) {
      mx = ov;
      mi = oi;
    }
  }
  float z = 0.f, zc = 0.f;
  for (int k = lane; k < K; k += 64) {
    const float p = fast_exp2((o[k] - mx) * kLog2e);
    z += p;
    zc = fmaf(p, centres[k], zc);
  }
  z = wave_sum(z);
  zc = wave_sum(zc);
  (void)red;
  if (lane == 0) {
    yhat[b] = zc / z;
    if (bin) bin[b] = mi;
  }
}

// order[rank(i)] = i with rank(i) = #{j : y_j < y_i or (y_j == y_i and j < i)}
__global__ __launch_bounds__(256) void sjf_order_kernel(const float* __restrict__ y, int B, int* __restrict__ order) {
  __shared__ float sy[1024];
  const int i = blockIdx.x * 256 + threadIdx.x;
  const float yi = i < B ? y[i] : 0.f;
  int rank = 0;
  for (int j0 = 0; j0 < B; j0 += 1024) {
    __syncthreads();
    for (int t = threadIdx.x; t < 1024; t += 256) sy[t] = (j0 + t < B) ? y[j0 + t] : 0.f;
    __syncthreads();
    const int jn = min(1024, B - j0);
    for (int t = 0; t < jn; ++t) {
      const float yj = sy[t];
      const int j = j0 + t;
      rank += (yj < yi || (yj == yi && j < i)) ? 1 : 0;
    }
  }
  if (i < B) order[rank] = i;
}

}  // namespace detail
}  // namespace estp

using namespace estp;
using namespace estp::detail;

extern "C" size_t estp_predict_workspace_size(int32_t B, int32_t d, int32_t hidden, int32_t K) {
  if (B < 1 || hidden < 1 || K < 1 || d < 1) return 0;
  const size_t nz = (size_t(d) + kKChunk - 1) / kKChunk;
  Carver c(nullptr);
  c.take<float>(nz * B * hidden);     // split-K partials of the first layer
  c.take<float>(size_t(B) * hidden);  // hidden activations
  c.take<float>(size_t(B) * K);       // head outputs
  return c.bytes();
}

extern "C" int estp_predict(const float* pooled, int32_t B, int32_t d, const float* W1, const float* b1,
                            int32_t hidden, int act, const float* W2, const float* b2, int32_t K,
                            const float* centres, float* yhat, int32_t* bin, int32_t* order, void* workspace,
                            size_t workspace_bytes, void* stream) {
  clear_error();
  ESTP_REQUIRE(pooled && W1 && W2 && yhat, ESTP_ERR_INVALID_ARG,
               "estp_predict: pooled, W1, W2 and yhat must be non-null");
  ESTP_REQUIRE(B >= 1 && B <= 65536 && d >= 1 && hidden >= 1 && K >= 1 && K <= 1024, ESTP_ERR_INVALID_ARG,
               "estp_predict: need 1 <= B <= 65536, d >= 1, hidden >= 1, 1 <= K <= 1024");
  ESTP_REQUIRE(K == 1 || centres, ESTP_ERR_INVALID_ARG, "estp_predict: centres required when K > 1");
  ESTP_REQUIRE(act == ESTP_ACT_RELU || act == ESTP_ACT_GELU_TANH, ESTP_ERR_INVALID_ARG,
               "estp_predict: unknown activation %d", act);
  const size_t need = estp_predict_workspace_size(B, d, hidden, K);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE, "estp_predict: workspace of %zu bytes, %zu needed",
               workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_predict: workspace must be non-null and 256-byte aligned");
  const int nz = (d + kKChunk - 1) / kKChunk;
  Carver c(workspace);
  float* part = c.take<float>(size_t(nz) * B * hidden);
  float* A = c.take<float>(size_t(B) * hidden);
  float* o = c.take<float>(size_t(B) * K);
  hipStream_t s = static_cast<hipStream_t>(stream);
  mlp_partial_kernel<<<dim3((hidden + kTH - 1) / kTH, (B + kTB - 1) / kTB, nz), dim3(256), 0, s>>>(pooled, W1, B, d,
                                                                                                 hidden, part);
  ESTP_CHECK_LAUNCH("mlp_partial_kernel");
  mlp_finish_kernel<<<dim3((size_t(B) * hidden + 255) / 256), dim3(256), 0, s>>>(part, b1, B, hidden, nz, act, A);
  ESTP_CHECK_LAUNCH("mlp_finish_kernel");
  head_out_kernel<<<dim3(B), dim3(256), 0, s>>>(A, W2, b2, centres, hidden, K, o, yhat, K > 1 ? bin : nullptr);
  ESTP_CHECK_LAUNCH("head_out_kernel");
  if (order) {
    sjf_order_kernel<<<dim3((B + 255) / 256), dim3(256), 0, s>>>(yhat, B, order);
    ESTP_CHECK_LAUNCH("sjf_order_kernel");
  }
  return ESTP_OK;
}
