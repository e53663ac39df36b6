// Attention importance, Eq. 1 (Section 4.1):
//   S_j = sum_l (1/N) sum_{i >= j} (1/Hq) sum_h A^{l,h}_{ij}
// with A the causal softmax of scale * q_i . k_j inside each prompt, without
// ever forming the N x N attention.
//
// Pass 1 (attn_lse_kernel) computes, for every (layer, query head, query row),
// the base-2 log-sum-exp of its causal score row.  Scores are formed on the
// matrix cores as S^T = K Q^T (keys on the MFMA "M" side, queries on "N"), so
// a lane owns one query column and 16 key rows of each 32 x 32 block and the
// row reduction over keys is a per-lane online max / sum.
//
// Pass 2 (attn_colsum_kernel) walks, for one 64-key block and one KV head,
// every later query block of every query head that shares that KV head
// (grouped-query reuse: the key fragments are loaded once and stay in
// registers), re-forms S = Q K^T (queries on "M", keys on "N"), and adds
// 2^(s2 - lse2) into per-lane column sums: a lane owns one key column and 16
// query rows, so the sum over queries is again per lane until a final
// two-step reduction (lane pair, then the four waves through LDS).  Partial
// column masses are written per (layer, KV head) and reduced in a fixed
// order by attn_reduce_kernel, which divides by N * Hq.  No atomics: results
// are bitwise reproducible.
#include "estp_common.h"

namespace estp {
namespace detail {

constexpr int kThreads = 256;
constexpr int kQBlock = 64;  // query rows per pass-1 workgroup
constexpr int kKBlock = 64;  // key columns per pass-2 workgroup

// Fragment of 8 consecutive bf16 of one row: row-major [*, row_stride] halves.
__device__ __forceinline__ bf16x8_t load_frag(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8_t*>(p);
}

// ---------------------------------------------------------------- pass 1
template <int DH>
__global__ __launch_bounds__(kThreads) void attn_lse_kernel(const uint16_t* __restrict__ Q,
                                                            const uint16_t* __restrict__ K,
                                                            const int* __restrict__ cu, int B, int n_tok,
                                                            int L, int Hq, int Hkv, int nqb_max, float c2,
                                                            float* __restrict__ lse2) {
  constexpr int KS = DH / 16;
  const int G = Hq / Hkv;
  // block -> (query block, prompt, layer * Hkv + kv head); largest query blocks first
  int idx = blockIdx.x;
  const int lg = idx % (L * Hkv);
  idx /= L * Hkv;
  const int b = idx % B;
  const int qblk = nqb_max - 1 - idx / B;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  if (qblk * kQBlock >= N) return;
  const int l = lg / Hkv, g = lg % Hkv;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 31;   // query column of this lane in a 32 x 32 block
  const int half = lane >> 5;  // which 8-wide k half of the fragment / which row quad of the output
  const size_t qrow = size_t(Hq) * DH, krow = size_t(Hkv) * DH;
  const uint16_t* Kl = K + size_t(l) * n_tok * krow + size_t(base) * krow + size_t(g) * DH;

  // units: (head in group, 32-row half of the query block), dealt to waves round-robin
  for (int u = wave; u < 2 * G; u += 4) {
    const int h = g * G + (u >> 1);
    const int q0 = qblk * kQBlock + (u & 1) * 32;
    if (q0 >= N) continue;
    const int qi = min(q0 + col, N - 1);
    const uint16_t* qp = Q + size_t(l) * n_tok * qrow + size_t(base + qi) * qrow + size_t(h) * DH + half * 8;
    bf16x8_t bq[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) bq[ks] = load_frag(qp + ks * 16);

    float m = -INFINITY, s = 0.f;
    const int q_last = q0 + col;  // this lane's query (may be >= N in a ragged tail)
    for (int kb = 0; kb <= q0 / 32; ++kb) {
      const int kj = min(kb * 32 + col, N - 1);
      const uint16_t* kp = Kl + size_t(kj) * krow + half * 8;
      f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(load_frag(kp + ks * 16), bq[ks], acc, 0, 0, 0);
      // acc[r]: key kb*32 + 8*(r/4) + 4*half + r%4, query q0 + col
      float z[16];
      float mx = -INFINITY;
      const bool diag = (kb == q0 / 32);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = kb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        z[r] = (!diag || j <= q_last) ? acc[r] * c2 : -INFINITY;
        mx = fmaxf(mx, z[r]);
      }
      const float mnew = fmaxf(m, mx);
      const float f = fast_exp2(fmaxf(m - mnew, kExp2Floor));
      s *= f;
#pragma unroll
      for (int r = 0; r < 16; ++r) s += fast_exp2(fmaxf(z[r] - mnew, kExp2Floor));
      m = mnew;
    }
    // lanes col and col + 32 hold the two row-quads of the same query column
    const float mo = __shfl_xor(m, 32, 64);
    const float so = __shfl_xor(s, 32, 64);
    const float M = fmaxf(m, mo);
    const float tot = s * fast_exp2(fmaxf(m - M, kExp2Floor)) + so * fast_exp2(fmaxf(mo - M, kExp2Floor));
    if (half == 0 && q0 + col < N)
      lse2[(size_t(l) * Hq + h) * n_tok + base + q0 + col] = M + fast_log2(tot);
  }
}

// ---------------------------------------------------------------- pass 2
template <int DH>
__global__ __launch_bounds__(kThreads) void attn_colsum_kernel(const uint16_t* __restrict__ Q,
                                                               const uint16_t* __restrict__ K,
                                                               const int* __restrict__ cu, int B, int n_tok,
                                                               int L, int Hq, int Hkv, float c2,
                                                               const float* __restrict__ lse2,
                                                               float* __restrict__ part) {
  constexpr int KS = DH / 16;
  __shared__ float red[4][kKBlock];
  const int G = Hq / Hkv;
  // block -> (key block, prompt, layer * Hkv + kv head); key block 0 (the most work) first
  int idx = blockIdx.x;
  const int lg = idx % (L * Hkv);
  idx /= L * Hkv;
  const int b = idx % B;
  const int kblk = idx / B;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  if (kblk * kKBlock >= N) return;
  const int l = lg / Hkv, g = lg % Hkv;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 31;   // key column of this lane in a 32 x 32 block
  const int half = lane >> 5;
  const size_t qrow = size_t(Hq) * DH, krow = size_t(Hkv) * DH;
  const uint16_t* Kl = K + size_t(l) * n_tok * krow + size_t(base) * krow + size_t(g) * DH;

  // key fragments of the two 32-key halves, resident for the whole walk
  bf16x8_t bk[2][KS];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int kj = min(kblk * kKBlock + cb * 32 + col, N - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) bk[cb][ks] = load_frag(Kl + size_t(kj) * krow + half * 8 + ks * 16);
  }
  float csum[2] = {0.f, 0.f};

  const int qb_first = kblk * (kKBlock / 32);
  const int qb_end = (N + 31) / 32;
  const int n_pairs = (qb_end - qb_first) * G;
  for (int p = wave; p < n_pairs; p += 4) {
    const int h = g * G + p % G;
    const int qb = qb_first + p / G;
    const int qi = min(qb * 32 + col, N - 1);
    const uint16_t* qp = Q + size_t(l) * n_tok * qrow + size_t(base + qi) * qrow + size_t(h) * DH + half * 8;
    bf16x8_t aq[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) aq[ks] = load_frag(qp + ks * 16);
    // lse of the 16 query rows this lane sees: rows qb*32 + 8*(r/4) + 4*half + r%4
    const float* lp = lse2 + (size_t(l) * Hq + h) * n_tok + base;
    float lr[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = qb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
      lr[r] = i < N ? lp[i] : INFINITY;  // rows past the prompt contribute 2^-inf = 0
    }
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      const int j = kblk * kKBlock + cb * 32 + col;  // this lane's key
      if (qb * 32 + 31 < kblk * kKBlock + cb * 32) continue;  // whole block above the diagonal
      f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq[ks], bk[cb][ks], acc, 0, 0, 0);
      float cs = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = qb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        const float pr = fast_exp2(fmaxf(fmaf(acc[r], c2, -lr[r]), kExp2Floor));
        cs += (j <= i) ? pr : 0.f;
      }
      csum[cb] += cs;
    }
  }
  // reduce: lane pair (the two row quads), then the four waves in fixed order
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) csum[cb] += __shfl_xor(csum[cb], 32, 64);
  if (half == 0) {
    red[wave][col] = csum[0];
    red[wave][32 + col] = csum[1];
  }
  __syncthreads();
  if (threadIdx.x < kKBlock) {
    const int t = threadIdx.x;
    const float v = ((red[0][t] + red[1][t]) + red[2][t]) + red[3][t];
    const int j = kblk * kKBlock + t;
    if (j < N) part[(size_t(l) * Hkv + g) * n_tok + base + j] = v;
  }
}

// S_j = (sum over layers and KV heads of the column masses) / (N * Hq)
__global__ __launch_bounds__(256) void attn_reduce_kernel(const float* __restrict__ part, const int* __restrict__ cu,
                                                          int n_tok, int LHkv, int Hq, float* __restrict__ S) {
  const int b = blockIdx.y;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= N) return;
  float v = 0.f;
  for (int k = 0; k < LHkv; ++k) v += part[size_t(k) * n_tok + base + j];
  S[base + j] = v / (float(N) * float(Hq));
}

template <int DH>
void launch(const uint16_t* Q, const uint16_t* K, const int* cu, int B, int max_seqlen, int n_tok, int L, int Hq,
            int Hkv, float scale, float* S, float* lse2, float* part, hipStream_t s) {
  const float c2 = scale * kLog2e;
  const int nqb = (max_seqlen + kQBlock - 1) / kQBlock;
  const int nkb = (max_seqlen + kKBlock - 1) / kKBlock;
  attn_lse_kernel<DH><<<dim3(size_t(nqb) * B * L * Hkv), dim3(kThreads), 0, s>>>(Q, K, cu, B, n_tok, L, Hq, Hkv, nqb, c2, lse2);
  attn_colsum_kernel<DH><<<dim3(size_t(nkb) * B * L * Hkv), dim3(kThreads), 0, s>>>(Q, K, cu, B, n_tok, L, Hq, Hkv, c2, lse2, part);
  attn_reduce_kernel<<<dim3((max_seqlen + 255) / 256, B), dim3(256), 0, s>>>(part, cu, n_tok, L * Hkv, Hq, S);
}

}  // namespace detail
}  // namespace estp

using namespace estp;
using namespace estp::detail;

extern "C" size_t estp_attn_importance_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t L,
                                                      int32_t Hq, int32_t Hkv, int32_t dh, int dtype) {
  (void)B;
  (void)max_seqlen;
  (void)dh;
  (void)dtype;
  if (n_tok < 1 || L < 1 || Hq < 1 || Hkv < 1) return 0;
  Carver c(nullptr);
  c.take<float>(size_t(L) * Hq * n_tok);   // lse2 [L, Hq, n_tok]
  c.take<float>(size_t(L) * Hkv * n_tok);  // column masses [L, Hkv, n_tok]
  return c.bytes();
}

extern "C" int estp_attn_importance(const void* Q, const void* K, const int32_t* cu_seqlens, int32_t B,
                                    int32_t max_seqlen, int64_t n_tok, int32_t L, int32_t Hq, int32_t Hkv,
                                    int32_t dh, float scale, int dtype, float* S, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  clear_error();
  ESTP_REQUIRE(Q && K && cu_seqlens && S, ESTP_ERR_INVALID_ARG,
               "estp_attn_importance: Q, K, cu_seqlens and S must be non-null");
  ESTP_REQUIRE(B >= 1 && max_seqlen >= 1 && L >= 1 && Hq >= 1 && Hkv >= 1, ESTP_ERR_INVALID_ARG,
               "estp_attn_importance: B, max_seqlen, L, Hq, Hkv must be >= 1");
  ESTP_REQUIRE(n_tok >= 1 && n_tok <= INT32_MAX, ESTP_ERR_INVALID_ARG,
               "estp_attn_importance: n_tok must be in [1, 2^31), got %lld", (long long)n_tok);
  ESTP_REQUIRE(max_seqlen <= n_tok, ESTP_ERR_INVALID_ARG, "estp_attn_importance: max_seqlen exceeds n_tok");
  ESTP_REQUIRE(Hq % Hkv == 0, ESTP_ERR_INVALID_ARG, "estp_attn_importance: Hq (%d) must be a multiple of Hkv (%d)",
               Hq, Hkv);
  ESTP_REQUIRE(scale > 0.f && scale < INFINITY, ESTP_ERR_INVALID_ARG,
               "estp_attn_importance: scale must be finite and > 0");
  ESTP_REQUIRE(dtype == ESTP_BF16 || dtype == ESTP_F32, ESTP_ERR_INVALID_ARG,
               "estp_attn_importance: unknown dtype %d", dtype);
  ESTP_REQUIRE(dtype == ESTP_BF16, ESTP_ERR_UNSUPPORTED,
               "estp_attn_importance: only ESTP_BF16 inputs are supported");
  ESTP_REQUIRE(dh == 32 || dh == 64 || dh == 128, ESTP_ERR_UNSUPPORTED,
               "estp_attn_importance: head_dim %d unsupported (32, 64, 128)", dh);
  ESTP_REQUIRE(aligned(Q, 16) && aligned(K, 16), ESTP_ERR_INVALID_ARG,
               "estp_attn_importance: Q and K must be 16-byte aligned");
  ESTP_REQUIRE(size_t(L) * Hq * n_tok < (size_t(1) << 40), ESTP_ERR_INVALID_ARG, "estp_attn_importance: too large");
  const size_t need = estp_attn_importance_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dtype);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_attn_importance: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_attn_importance: workspace must be non-null and 256-byte aligned");

  Carver c(workspace);
  float* lse2 = c.take<float>(size_t(L) * Hq * n_tok);
  float* part = c.take<float>(size_t(L) * Hkv * n_tok);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint16_t* q = static_cast<const uint16_t*>(Q);
  const uint16_t* k = static_cast<const uint16_t*>(K);
  const int n = int(n_tok);
  switch (dh) {
    case 32: launch<32>(q, k, cu_seqlens, B, max_seqlen, n, L, Hq, Hkv, scale, S, lse2, part, s); break;
    case 64: launch<64>(q, k, cu_seqlens, B, max_seqlen, n, L, Hq, Hkv, scale, S, lse2, part, s); break;
    default: launch<128>(q, k, cu_seqlens, B, max_seqlen, n, L, Hq, Hkv, scale, S, lse2, part, s); break;
  }
  ESTP_CHECK_LAUNCH("estp_attn_importance");
  return ESTP_OK;
}
