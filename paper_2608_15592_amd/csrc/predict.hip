// Length head (Section 4.3) and shortest-job-first order (Section 5.4).
//
//   a = act(W1 h + b1)            mlp_partial_kernel (split-K fp32 tiles) + mlp_finish_kernel
//   o = W2 a + b2                 head_out_kernel: one workgroup per prompt
//   K == 1: yhat = o_0;  K > 1: p = softmax(o), yhat = sum_k p_k c_k (Eq. 7), bin = argmax p
//   order: stable ascending argsort of yhat (rank counting, exact and deterministic)
//
// One training step of the K-bin head (Eq. 6 - Eq. 8, AdamW as in Section 5.1):
//   forward as above, keeping the pre-activations  mlp_partial_kernel + train_hidden_kernel
//   Eq. 6 soft labels, Eq. 8 loss, dL/do per sample  train_out_kernel (one workgroup per sample)
//   dL/dz = (dL/do W2) act'(z)                       train_dz_kernel
//   gradients of b1, W2, b2 and their AdamW update   train_update_small_kernel
//   gradient of W1 and its AdamW update, fused       train_update_w1_kernel
// Every batch sum runs in a fixed order: the step is bitwise reproducible.
#include <cmath>

#include "estp_common.h"

namespace estp {
namespace detail {

constexpr int kTB = 32;     // prompts per tile
constexpr int kTH = 32;     // hidden units per tile
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
// hundreds of workgroups even for small batches.  The whole 256-deep chunk of both
// operands goes into LDS in one round (all loads in flight together, 16 bytes each
// when rows allow it), stored k-major so that the compute loop reads without bank
// conflicts; each output is then summed over k in order.
template <bool kVec>
__global__ __launch_bounds__(256) void mlp_partial_kernel(const float* __restrict__ P, const float* __restrict__ W1,
                                                          int B, int d, int Hd, float* __restrict__ part) {
  __shared__ float sp[kKChunk][kTB + 1];
  __shared__ float sw[kKChunk][kTH + 1];
  const int th = blockIdx.x * kTH, tb = blockIdx.y * kTB, z = blockIdx.z;
  const int k_lo = z * kKChunk, nk = min(d, k_lo + kKChunk) - k_lo;
  const int tx = threadIdx.x & 31;         // hidden unit in the tile
  const int ty = (threadIdx.x >> 5) * 4;   // first of 4 prompts
  if (kVec) {
    // lane (r = lane % 32, h = lane / 32) of wave w loads 16 bytes of row r at depth 4 (2 (w + 4 q) + h)
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 31, h = lane >> 5;
    float4 vp[8], vw[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int k4 = (2 * (wave + 4 * q) + h) * 4;
      const bool kin = k4 < nk;  // nk is a multiple of 4 here
      vp[q] = (tb + r < B && kin) ? *reinterpret_cast<const float4*>(P + size_t(tb + r) * d + k_lo + k4)
                                  : float4{0.f, 0.f, 0.f, 0.f};
      vw[q] = (th + r < Hd && kin) ? *reinterpret_cast<const float4*>(W1 + size_t(th + r) * d + k_lo + k4)
                                   : float4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int k4 = (2 * (wave + 4 * q) + h) * 4;
      sp[k4][r] = vp[q].x;
      sp[k4 + 1][r] = vp[q].y;
      sp[k4 + 2][r] = vp[q].z;
      sp[k4 + 3][r] = vp[q].w;
      sw[k4][r] = vw[q].x;
      sw[k4 + 1][r] = vw[q].y;
      sw[k4 + 2][r] = vw[q].z;
      sw[k4 + 3][r] = vw[q].w;
    }
  } else {
    for (int e = threadIdx.x; e < kTB * kKChunk; e += 256) {
      const int r = e / kKChunk, k = e % kKChunk;  // consecutive threads read consecutive k of one row
      sp[k][r] = (tb + r < B && k < nk) ? P[size_t(tb + r) * d + k_lo + k] : 0.f;
      sw[k][r] = (th + r < Hd && k < nk) ? W1[size_t(th + r) * d + k_lo + k] : 0.f;
    }
  }
  __syncthreads();
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int k = 0; k < nk; ++k) {
    const float w = sw[k][tx];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = fmaf(sp[k][ty + i], w, acc[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int b = tb + ty + i, j = th + tx;
    if (b < B && j < Hd) part[(size_t(z) * B + b) * Hd + j] = acc[i];
  }
}

// Launch of the split-K partials: 16-byte loads when every row starts 16-byte aligned.
void launch_mlp_partial(const float* P, const float* W1, int B, int d, int Hd, float* part, hipStream_t s) {
  const dim3 grid((Hd + kTH - 1) / kTH, (B + kTB - 1) / kTB, (d + kKChunk - 1) / kKChunk);
  if (d % 4 == 0 && aligned(P, 16) && aligned(W1, 16))
    mlp_partial_kernel<true><<<grid, dim3(256), 0, s>>>(P, W1, B, d, Hd, part);
  else
    mlp_partial_kernel<false><<<grid, dim3(256), 0, s>>>(P, W1, B, d, Hd, part);
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

// ---------------------------------------------------------------- training step

__device__ __forceinline__ float act_grad(float z, int act) {
  if (act == ESTP_ACT_RELU) return z > 0.f ? 1.f : 0.f;
  const float k = 0.7978845608028654f;  // sqrt(2 / pi)
  const float t = tanhf(k * fmaf(0.044715f * z, z * z, z));
  return 0.5f * (1.f + t) + 0.5f * z * (1.f - t * t) * k * fmaf(3.f * 0.044715f, z * z, 1.f);
}

struct AdamW {
  float lr, beta1, beta2, eps, decay;  // decay = 1 - lr * weight_decay
  float bc1, bc2;                      // 1 / (1 - beta1^t), 1 / (1 - beta2^t)
};

__device__ __forceinline__ void adamw_update(float& th, float& m, float& v, float g, const AdamW& a) {
  m = fmaf(a.beta1, m, (1.f - a.beta1) * g);
  v = fmaf(a.beta2, v, (1.f - a.beta2) * g * g);
  th = th * a.decay - a.lr * (m * a.bc1) / (sqrtf(v * a.bc2) + a.eps);
}

// Z[b, j] = sum_z part[z, b, j] + b1[j] (kept for the backward pass), A = act(Z).
__global__ __launch_bounds__(256) void train_hidden_kernel(const float* __restrict__ part,
                                                           const float* __restrict__ b1, int B, int Hd, int nz,
                                                           int act, float* __restrict__ Z, float* __restrict__ A) {
  const size_t e = size_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= size_t(B) * Hd) return;
  float v = 0.f;
  for (int z = 0; z < nz; ++z) v += part[size_t(z) * B * Hd + e];
  v += b1[e % Hd];
  Z[e] = v;
  A[e] = act_fn(v, act);
}

// One workgroup (256 threads) per sample b: o = W2 a + b2, p-hat = softmax(o),
// y-hat = sum_k p-hat_k c_k (Eq. 7); the true bin i of y (edges, Eq. 6), the soft
// labels p_j = exp(-|j - i|) / sum_k exp(-|k - i|); the sample's loss
// lambda3 CE(p, p-hat) + (1 - lambda3) (y - y-hat)^2 (Eq. 8) and
// dL/do_k = (lambda3 (p-hat_k - p_k) - 2 (1 - lambda3) (y - y-hat) p-hat_k (c_k - y-hat)) / B.
__global__ __launch_bounds__(256) void train_out_kernel(const float* __restrict__ A, const float* __restrict__ W2,
                                                        const float* __restrict__ b2,
                                                        const float* __restrict__ edges,
                                                        const float* __restrict__ centres,
                                                        const float* __restrict__ y, int B, int Hd, int K,
                                                        float lambda3, float* __restrict__ o_ws,
                                                        float* __restrict__ dO, float* __restrict__ loss_b) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* a = A + size_t(b) * Hd;
  float* o = o_ws + size_t(b) * K;
  for (int k = wave; k < K; k += 4) {  // one wave per output, lanes over the hidden units
    const float* w = W2 + size_t(k) * Hd;
    float v = 0.f;
    for (int j = lane; j < Hd; j += 64) v = fmaf(w[j], a[j], v);
    v = wave_sum(v);
    if (lane == 0) o[k] = v + b2[k];
  }
  __syncthreads();
  if (wave != 0) return;
  const float yb = y[b];
  float mx = -INFINITY;
  int below = 0;  // edges 1 .. K-1 at or below y: the bin index
  for (int k = lane; k < K; k += 64) {
    mx = fmaxf(mx, o[k]);
    if (k >= 1 && edges[k] <= yb) ++below;
  }
  mx = wave_max(mx);
  const int i = int(wave_sum(float(below)));
  float z = 0.f, zc = 0.f, zs = 0.f;
  for (int k = lane; k < K; k += 64) {
    const float q = fast_exp2((o[k] - mx) * kLog2e);
    z += q;
    zc = fmaf(q, centres[k], zc);
    zs += expf(-fabsf(float(k - i)));
  }
  z = wave_sum(z);
  zc = wave_sum(zc);
  zs = wave_sum(zs);
  const float lse = mx + logf(z);
  const float yhat = zc / z;
  const float r = yb - yhat;
  float ce = 0.f;
  for (int k = lane; k < K; k += 64) {
    const float ph = fast_exp2((o[k] - lse) * kLog2e);
    const float pk = expf(-fabsf(float(k - i))) / zs;
    ce = fmaf(-pk, o[k] - lse, ce);
    const float g = lambda3 * (ph - pk) - 2.f * (1.f - lambda3) * r * ph * (centres[k] - yhat);
    dO[size_t(b) * K + k] = g / float(B);
  }
  ce = wave_sum(ce);
  if (lane == 0) loss_b[b] = lambda3 * ce + (1.f - lambda3) * r * r;
}

// loss = (1/B) sum_b loss_b, in a fixed order (strided per thread, then a fixed tree).
__global__ __launch_bounds__(256) void train_loss_kernel(const float* __restrict__ loss_b, int B,
                                                         float* __restrict__ loss) {
  __shared__ float sh[4];
  float v = 0.f;
  for (int b = threadIdx.x; b < B; b += 256) v += loss_b[b];
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) *loss = (sh[0] + sh[1] + sh[2] + sh[3]) / float(B);
}

// dZ[b, j] = (sum_k dO[b, k] W2[k, j]) act'(Z[b, j])
__global__ __launch_bounds__(256) void train_dz_kernel(const float* __restrict__ dO, const float* __restrict__ W2,
                                                       const float* __restrict__ Z, int B, int Hd, int K, int act,
                                                       float* __restrict__ dZ) {
  const size_t e = size_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= size_t(B) * Hd) return;
  const int b = int(e / Hd), j = int(e % Hd);
  float g = 0.f;
  for (int k = 0; k < K; ++k) g = fmaf(dO[size_t(b) * K + k], W2[size_t(k) * Hd + j], g);
  dZ[e] = g * act_grad(Z[e], act);
}

// Gradients of b1 [Hd], W2 [K, Hd], b2 [K] (sums over the batch in order) and their
// AdamW updates.  th/m/v point at b1 of the flat parameter layout: b1, then W2, then b2.
__global__ __launch_bounds__(256) void train_update_small_kernel(const float* __restrict__ dZ,
                                                                 const float* __restrict__ dO,
                                                                 const float* __restrict__ A, int B, int Hd, int K,
                                                                 float* __restrict__ th, float* __restrict__ m,
                                                                 float* __restrict__ v, AdamW opt) {
  const size_t e = size_t(blockIdx.x) * 256 + threadIdx.x;
  const size_t n_w2 = size_t(K) * Hd;
  if (e >= size_t(Hd) + n_w2 + K) return;
  float g = 0.f;
  if (e < size_t(Hd)) {
    for (int b = 0; b < B; ++b) g += dZ[size_t(b) * Hd + e];
  } else if (e < size_t(Hd) + n_w2) {
    const size_t w = e - Hd;
    const int k = int(w / Hd), j = int(w % Hd);
    for (int b = 0; b < B; ++b) g = fmaf(dO[size_t(b) * K + k], A[size_t(b) * Hd + j], g);
  } else {
    const int k = int(e - Hd - n_w2);
    for (int b = 0; b < B; ++b) g += dO[size_t(b) * K + k];
  }
  float t = th[e], mm = m[e], vv = v[e];
  adamw_update(t, mm, vv, g, opt);
  th[e] = t;
  m[e] = mm;
  v[e] = vv;
}

// W1 [Hd, d]: g[j, c] = sum_b dZ[b, j] P[b, c] and its AdamW update, fused.  A workgroup
// covers 1024 consecutive features of one row j (4 per thread, 16-byte accesses).
__global__ __launch_bounds__(256) void train_update_w1_kernel(const float* __restrict__ dZ,
                                                              const float* __restrict__ P, int B, int d, int Hd,
                                                              float* __restrict__ W1, float* __restrict__ m,
                                                              float* __restrict__ v, AdamW opt) {
  const int j = blockIdx.y;
  const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (c >= d) return;
  float4 g = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int b = 0; b < B; ++b) {
    const float w = dZ[size_t(b) * Hd + j];
    const float4 p = *reinterpret_cast<const float4*>(P + size_t(b) * d + c);
    g.x = fmaf(w, p.x, g.x);
    g.y = fmaf(w, p.y, g.y);
    g.z = fmaf(w, p.z, g.z);
    g.w = fmaf(w, p.w, g.w);
  }
  const size_t o = size_t(j) * d + c;
  float4 t = *reinterpret_cast<const float4*>(W1 + o);
  float4 mm = *reinterpret_cast<const float4*>(m + o);
  float4 vv = *reinterpret_cast<const float4*>(v + o);
  adamw_update(t.x, mm.x, vv.x, g.x, opt);
  adamw_update(t.y, mm.y, vv.y, g.y, opt);
  adamw_update(t.z, mm.z, vv.z, g.z, opt);
  adamw_update(t.w, mm.w, vv.w, g.w, opt);
  *reinterpret_cast<float4*>(W1 + o) = t;
  *reinterpret_cast<float4*>(m + o) = mm;
  *reinterpret_cast<float4*>(v + o) = vv;
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
  launch_mlp_partial(pooled, W1, B, d, hidden, part, s);
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

extern "C" size_t estp_head_train_step_workspace_size(int32_t B, int32_t d, int32_t hidden, int32_t K) {
  if (B < 1 || hidden < 1 || K < 1 || d < 1) return 0;
  const size_t nz = (size_t(d) + kKChunk - 1) / kKChunk;
  Carver c(nullptr);
  c.take<float>(nz * B * hidden);     // split-K partials of the first layer
  c.take<float>(size_t(B) * hidden);  // pre-activations Z
  c.take<float>(size_t(B) * hidden);  // activations A
  c.take<float>(size_t(B) * hidden);  // dL/dZ
  c.take<float>(size_t(B) * K);       // head outputs
  c.take<float>(size_t(B) * K);       // dL/do
  c.take<float>(size_t(B));           // per-sample losses
  c.take<float>(1);                   // batch loss when the caller passes none
  return c.bytes();
}

extern "C" int estp_head_train_step(const float* pooled, const float* y, int32_t B, int32_t d, int32_t hidden,
                                    int32_t K, int act, const float* edges, const float* centres, float* theta,
                                    float* m, float* v, int32_t step, float lambda3, float lr, float beta1,
                                    float beta2, float eps, float weight_decay, float* loss, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  clear_error();
  ESTP_REQUIRE(pooled && y && edges && centres && theta && m && v, ESTP_ERR_INVALID_ARG,
               "estp_head_train_step: pooled, y, edges, centres, theta, m and v must be non-null");
  ESTP_REQUIRE(B >= 1 && B <= 65536 && hidden >= 1 && K >= 2 && K <= 1024, ESTP_ERR_INVALID_ARG,
               "estp_head_train_step: need 1 <= B <= 65536, hidden >= 1, 2 <= K <= 1024");
  ESTP_REQUIRE(d >= 4 && d % 4 == 0, ESTP_ERR_INVALID_ARG,
               "estp_head_train_step: d must be a positive multiple of 4, got %d", d);
  ESTP_REQUIRE(act == ESTP_ACT_RELU || act == ESTP_ACT_GELU_TANH, ESTP_ERR_INVALID_ARG,
               "estp_head_train_step: unknown activation %d", act);
  ESTP_REQUIRE(step >= 1, ESTP_ERR_INVALID_ARG, "estp_head_train_step: step counts from 1, got %d", step);
  ESTP_REQUIRE(lambda3 >= 0.f && lambda3 <= 1.f, ESTP_ERR_INVALID_ARG,
               "estp_head_train_step: lambda3 must be in [0, 1]");
  ESTP_REQUIRE(lr >= 0.f && lr < INFINITY && weight_decay >= 0.f && weight_decay < INFINITY && eps > 0.f &&
                   eps < INFINITY,
               ESTP_ERR_INVALID_ARG, "estp_head_train_step: need finite lr >= 0, weight_decay >= 0, eps > 0");
  ESTP_REQUIRE(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f, ESTP_ERR_INVALID_ARG,
               "estp_head_train_step: betas must be in [0, 1)");
  ESTP_REQUIRE(aligned(pooled, 16) && aligned(theta, 16) && aligned(m, 16) && aligned(v, 16), ESTP_ERR_INVALID_ARG,
               "estp_head_train_step: pooled, theta, m and v must be 16-byte aligned");
  const size_t need = estp_head_train_step_workspace_size(B, d, hidden, K);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_head_train_step: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_head_train_step: workspace must be non-null and 256-byte aligned");

  const int nz = (d + kKChunk - 1) / kKChunk;
  Carver c(workspace);
  float* part = c.take<float>(size_t(nz) * B * hidden);
  float* Z = c.take<float>(size_t(B) * hidden);
  float* A = c.take<float>(size_t(B) * hidden);
  float* dZ = c.take<float>(size_t(B) * hidden);
  float* o = c.take<float>(size_t(B) * K);
  float* dO = c.take<float>(size_t(B) * K);
  float* loss_b = c.take<float>(size_t(B));
  float* loss_ws = c.take<float>(1);
  float* W1 = theta;
  float* b1 = W1 + size_t(hidden) * d;
  float* W2 = b1 + hidden;
  float* b2 = W2 + size_t(K) * hidden;
  AdamW opt;
  opt.lr = lr;
  opt.beta1 = beta1;
  opt.beta2 = beta2;
  opt.eps = eps;
  opt.decay = float(1.0 - double(lr) * double(weight_decay));
  opt.bc1 = float(1.0 / (1.0 - std::pow(double(beta1), double(step))));
  opt.bc2 = float(1.0 / (1.0 - std::pow(double(beta2), double(step))));
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t nbh = size_t(B) * hidden;
  launch_mlp_partial(pooled, W1, B, d, hidden, part, s);
  ESTP_CHECK_LAUNCH("mlp_partial_kernel");
  train_hidden_kernel<<<dim3((nbh + 255) / 256), dim3(256), 0, s>>>(part, b1, B, hidden, nz, act, Z, A);
  ESTP_CHECK_LAUNCH("train_hidden_kernel");
  train_out_kernel<<<dim3(B), dim3(256), 0, s>>>(A, W2, b2, edges, centres, y, B, hidden, K, lambda3, o, dO, loss_b);
  ESTP_CHECK_LAUNCH("train_out_kernel");
  train_loss_kernel<<<dim3(1), dim3(256), 0, s>>>(loss_b, B, loss ? loss : loss_ws);
  ESTP_CHECK_LAUNCH("train_loss_kernel");
  train_dz_kernel<<<dim3((nbh + 255) / 256), dim3(256), 0, s>>>(dO, W2, Z, B, hidden, K, act, dZ);
  ESTP_CHECK_LAUNCH("train_dz_kernel");
  const size_t n_small = size_t(hidden) + size_t(K) * hidden + K;
  const size_t off_b1 = size_t(hidden) * d;
  train_update_small_kernel<<<dim3((n_small + 255) / 256), dim3(256), 0, s>>>(dZ, dO, A, B, hidden, K, theta + off_b1,
                                                                              m + off_b1, v + off_b1, opt);
  ESTP_CHECK_LAUNCH("train_update_small_kernel");
  train_update_w1_kernel<<<dim3((d / 4 + 255) / 256, hidden), dim3(256), 0, s>>>(dZ, pooled, B, d, hidden, W1, m, v,
                                                                                 opt);
  ESTP_CHECK_LAUNCH("train_update_w1_kernel");
  return ESTP_OK;
}
