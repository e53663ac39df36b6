// Analyses on the path's outputs.
//
// Entropy / semantics misalignment (the diagnostic behind Fig. 1b, Section 1):
// within each prompt the tokens are ranked by H and by S (ascending, equal
// values by token index) and split into the lowest floor(f_low N) and the
// highest floor(f_high N).  misalignment_kernel (one workgroup per prompt)
// finds the four split keys by radix selection over 64-bit keys
// (order-preserving float bits, token index) in eight 8-bit passes each, then
// counts (#high-H, #high-H that are low-S, #low-H, #low-H that are high-S).
// Integer counts: exact and bitwise reproducible.
//
// Static shortest-job-first batches (Section 5.4): requests taken in a given
// order (the SJF order of the predicted lengths, say) form batches of `batch`;
// each batch runs for its longest true length, batches back to back.
// sjf_padding_kernel (one workgroup) returns the padded tokens, the useful
// tokens and the sum of completion times start(batch) + y_i, in int64.
#include "estp_common.h"

namespace estp {
namespace detail {

constexpr int kAThreads = 256;

__device__ __forceinline__ uint64_t rank_key(float v, int i) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // monotone in v
  return (uint64_t(u) << 32) | uint32_t(i);
}

// The key of rank r (0-based) among the prompt's N keys, by 8-bit radix selection.
__device__ uint64_t select_rank(const float* __restrict__ v, int N, int r, int* hist, uint64_t* sh_prefix,
                                int* sh_r) {
  uint64_t prefix = 0, mask = 0;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int k = threadIdx.x; k < 256; k += kAThreads) hist[k] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < N; i += kAThreads) {
      const uint64_t key = rank_key(v[i], i);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int rr = r, d = 0;
      while (d < 255 && rr >= hist[d]) rr -= hist[d++];
      *sh_prefix = prefix | (uint64_t(d) << shift);
      *sh_r = rr;
    }
    __syncthreads();
    prefix = *sh_prefix;
    r = *sh_r;
    mask |= uint64_t(255) << shift;
    __syncthreads();
  }
  return prefix;
}

__global__ __launch_bounds__(kAThreads) void misalignment_kernel(const float* __restrict__ H,
                                                                 const float* __restrict__ S,
                                                                 const int* __restrict__ cu, float f_low,
                                                                 float f_high, int* __restrict__ counts) {
  __shared__ int hist[256];
  __shared__ uint64_t sh_prefix;
  __shared__ int sh_r;
  __shared__ int red[4][kAThreads / 64];
  const int b = blockIdx.x;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const int nl = int(floorf(f_low * float(N))), nh = int(floorf(f_high * float(N)));
  const float* h = H + base;
  const float* s = S + base;
  // low set: key < key of rank nl (empty when nl = 0); high set: key >= key of rank N - nh (empty when nh = 0)
  const uint64_t hl = nl > 0 ? select_rank(h, N, nl < N ? nl : N - 1, hist, &sh_prefix, &sh_r) : 0;
  const uint64_t hh = nh > 0 ? select_rank(h, N, N - nh, hist, &sh_prefix, &sh_r) : 0;
  const uint64_t sl = nl > 0 ? select_rank(s, N, nl < N ? nl : N - 1, hist, &sh_prefix, &sh_r) : 0;
  const uint64_t sh = nh > 0 ? select_rank(s, N, N - nh, hist, &sh_prefix, &sh_r) : 0;
  int c[4] = {0, 0, 0, 0};
  for (int i = threadIdx.x; i < N; i += kAThreads) {
    const uint64_t kh = rank_key(h[i], i), ks = rank_key(s[i], i);
    // nl = N puts every token low (the selected rank N - 1 is then itself included)
    const bool lowH = nl > 0 && (kh < hl || (nl == N));
    const bool lowS = nl > 0 && (ks < sl || (nl == N));
    const bool highH = nh > 0 && kh >= hh;
    const bool highS = nh > 0 && ks >= sh;
    c[0] += highH;
    c[1] += highH && lowS;
    c[2] += lowH;
    c[3] += lowH && highS;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int v = c[q];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) red[q][wave] = v;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    int v = 0;
    for (int w = 0; w < kAThreads / 64; ++w) v += red[threadIdx.x][w];
    counts[size_t(b) * 4 + threadIdx.x] = v;
  }
}

__global__ __launch_bounds__(kAThreads) void sjf_padding_kernel(const int* __restrict__ y,
                                                                const int* __restrict__ order, int B, int batch,
                                                                long long* __restrict__ out) {
  __shared__ long long off[kAThreads];
  __shared__ long long red[3][kAThreads];
  const int nb = (B + batch - 1) / batch;
  const int per = (nb + kAThreads - 1) / kAThreads;
  const int k0 = threadIdx.x * per, k1 = min(nb, k0 + per);
  auto member = [&](int p) { return y[order ? order[p] : p]; };
  // pass 1: this thread's batches' maxima, for the start offsets
  long long span = 0;
  for (int k = k0; k < k1; ++k) {
    int mx = 0;
    for (int p = k * batch; p < min(B, (k + 1) * batch); ++p) mx = max(mx, member(p));
    span += mx;
  }
  off[threadIdx.x] = span;
  __syncthreads();
  if (threadIdx.x == 0) {  // exclusive scan, in order
    long long run = 0;
    for (int t = 0; t < kAThreads; ++t) {
      const long long v = off[t];
      off[t] = run;
      run += v;
    }
  }
  __syncthreads();
  // pass 2: padding, useful tokens and completion times of this thread's batches
  long long start = off[threadIdx.x], padded = 0, useful = 0, jct = 0;
  for (int k = k0; k < k1; ++k) {
    int mx = 0;
    long long sum = 0;
    const int p1 = min(B, (k + 1) * batch);
    for (int p = k * batch; p < p1; ++p) {
      const int v = member(p);
      mx = max(mx, v);
      sum += v;
    }
    const long long size = p1 - k * batch;
    padded += size * mx - sum;
    useful += sum;
    jct += size * start + sum;
    start += mx;
  }
  red[0][threadIdx.x] = padded;
  red[1][threadIdx.x] = useful;
  red[2][threadIdx.x] = jct;
  __syncthreads();
  if (threadIdx.x < 3) {
    long long v = 0;
    for (int t = 0; t < kAThreads; ++t) v += red[threadIdx.x][t];
    out[threadIdx.x] = v;
  }
}

}  // namespace detail
}  // namespace estp

using namespace estp;
using namespace estp::detail;

extern "C" int estp_misalignment(const float* H, const float* S, const int32_t* cu_seqlens, int32_t B,
                                 float frac_low, float frac_high, int32_t* counts, void* stream) {
  clear_error();
  ESTP_REQUIRE(H && S && cu_seqlens && counts, ESTP_ERR_INVALID_ARG,
               "estp_misalignment: H, S, cu_seqlens and counts must be non-null");
  ESTP_REQUIRE(B >= 1, ESTP_ERR_INVALID_ARG, "estp_misalignment: B must be >= 1");
  ESTP_REQUIRE(frac_low >= 0.f && frac_low <= 1.f && frac_high >= 0.f && frac_high <= 1.f, ESTP_ERR_INVALID_ARG,
               "estp_misalignment: fractions must be in [0, 1]");
  ESTP_REQUIRE(fits_launch(size_t(B), kAThreads), ESTP_ERR_UNSUPPORTED,
               "estp_misalignment: B = %d is more than one launch holds", B);
  if (debug_checks_enabled()) {
    const int st = debug_check_cu("estp_misalignment", cu_seqlens, B, -1, INT32_MAX, static_cast<hipStream_t>(stream),
                                  nullptr);
    if (st != ESTP_OK) return st;
  }
  misalignment_kernel<<<dim3(B), dim3(kAThreads), 0, static_cast<hipStream_t>(stream)>>>(H, S, cu_seqlens, frac_low,
                                                                                         frac_high, counts);
  ESTP_CHECK_LAUNCH("misalignment_kernel");
  return ESTP_OK;
}

extern "C" int estp_sjf_padding(const int32_t* lengths, const int32_t* order, int32_t B, int32_t batch,
                                int64_t* out, void* stream) {
  clear_error();
  ESTP_REQUIRE(lengths && out, ESTP_ERR_INVALID_ARG, "estp_sjf_padding: lengths and out must be non-null");
  ESTP_REQUIRE(B >= 1 && batch >= 1, ESTP_ERR_INVALID_ARG, "estp_sjf_padding: B and batch must be >= 1");
  sjf_padding_kernel<<<dim3(1), dim3(kAThreads), 0, static_cast<hipStream_t>(stream)>>>(
      lengths, order, B, batch, reinterpret_cast<long long*>(out));
  ESTP_CHECK_LAUNCH("sjf_padding_kernel");
  return ESTP_OK;
}
