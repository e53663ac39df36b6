// Attention importance (Eq. 1, Section 4.1) for fp32 queries and keys, with
// fp32 arithmetic throughout: the same two passes, block list and
// intermediate layouts as the bf16 matrix-core kernels, as register-tiled
// VALU dot products.
//
// Pass 1 (attn_lse_f32_kernel): one workgroup per (half of a 256-query
// block, layer, query head).  Its 128 queries stay in LDS (k-major) for the
// whole walk; the prompt's keys stream through a double-buffered k-major LDS
// tile of 64 (loaded into registers one tile ahead).  Thread (tk, tq) forms
// the 8 x 4 scores of keys 4tk..4tk+3, 32+4tk..32+4tk+3 and queries
// 4tq..4tq+3 of each tile (three float4 LDS reads per 32 FMAs), masks keys
// after their query and folds them into an exact online log-sum-exp per
// query in base 2.  The 8 threads that share a query merge at the end:
// lse2 = log2 sum_j 2^(c s_ij), c = scale * log2 e.
//
// Pass 2 (attn_colsum_f32_kernel): one workgroup per (half of a 256-key
// block, layer, KV head).  Its 128 keys stay in LDS; every later 64-query
// tile of each query head of the group streams through, with the tile's row
// lse2.  Thread (tq, tk) forms the 8 x 4 scores of queries 4tq..4tq+3,
// 32+4tq..32+4tq+3 and keys 4tk..4tk+3 and adds 2^(c s_ij - lse2_i) over the
// queries i >= j (i > j when the diagonal is left out) to its keys' column
// masses; the 8 threads that share a key add theirs in a fixed order.
// attn_reduce_kernel then divides by N * Hq as for the bf16 path.  No
// atomics: bitwise reproducible.
#include "estp_common.h"
#include "f32_paths.h"

namespace estp {
namespace detail {
namespace {

constexpr int kGThreads = 256;
constexpr int kGRows = 128;  // queries (pass 1) or keys (pass 2) of one workgroup: half a 256-row block
constexpr int kGTile = 64;   // streamed keys (pass 1) or queries (pass 2) per LDS tile
constexpr int kGPad = 4;     // row-pitch padding of the k-major LDS tiles; keeps float4 alignment

// ROWS rows of DH floats moved into LDS k-major (element (row r, feature c) at
// c * kPitch + r).  Each thread carries kPer float4 of the rows, read row-major
// from global memory (consecutive threads, consecutive 16-byte pieces of a row).
template <int DH, int ROWS>
struct KMajor {
  static constexpr int kPitch = ROWS + kGPad;
  static constexpr int kPer = ROWS * DH / 4 / kGThreads;
  static_assert(kPer >= 1 && ROWS * DH / 4 == kPer * kGThreads, "load pattern");
  float4 v[kPer];
  // row r of the tile from rowptr(r), a valid (clamped) row
  template <class RowPtr>
  __device__ __forceinline__ void load(int tid, RowPtr rowptr) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = tid + kGThreads * i;
      v[i] = *reinterpret_cast<const float4*>(rowptr(idx / (DH / 4)) + 4 * (idx % (DH / 4)));
    }
  }
  __device__ __forceinline__ void store(int tid, float* lds) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = tid + kGThreads * i;
      const int r = idx / (DH / 4), c = 4 * (idx % (DH / 4));
      lds[(c + 0) * kPitch + r] = v[i].x;
      lds[(c + 1) * kPitch + r] = v[i].y;
      lds[(c + 2) * kPitch + r] = v[i].z;
      lds[(c + 3) * kPitch + r] = v[i].w;
    }
  }
};

// sc[i][j] = sum_c a_i[c] b_j[c] for the thread's 8 "a" rows (a0 .. a0 + 3 and
// a0 + 32 .. a0 + 35 of a k-major tile of pitch PA) and 4 "b" rows (b0 .. b0 + 3
// of a k-major tile of pitch PB)
template <int DH, int PA, int PB>
__device__ __forceinline__ void scores_8x4(const float* __restrict__ a, int a0, const float* __restrict__ b, int b0,
                                           float (&sc)[8][4]) {
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) sc[i][j] = 0.f;
#pragma unroll 8
  for (int c = 0; c < DH; ++c) {
    const float4 x0 = *reinterpret_cast<const float4*>(a + c * PA + a0);
    const float4 x1 = *reinterpret_cast<const float4*>(a + c * PA + a0 + 32);
    const float4 y = *reinterpret_cast<const float4*>(b + c * PB + b0);
    const float av[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    const float bv[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) sc[i][j] = fmaf(av[i], bv[j], sc[i][j]);
  }
}

// (m, s) with s = sum 2^(x - m): the state of both
__device__ __forceinline__ void lse_merge(float& m, float& s, float mo, float so) {
  const float M = fmaxf(m, mo);
  s = s * fast_exp2(fmaxf(m - M, kExp2Floor)) + so * fast_exp2(fmaxf(mo - M, kExp2Floor));
  m = M;
}

}  // namespace

template <int DH>
__global__ __launch_bounds__(kGThreads) void attn_lse_f32_kernel(const float* __restrict__ Q,
                                                                 const float* __restrict__ K,
                                                                 const int* __restrict__ cu, int B, int n_tok, int L,
                                                                 int Hq, int Hkv, int nqb_max, float c2,
                                                                 const int2* __restrict__ blist,
                                                                 float* __restrict__ lse2) {
  using QT = KMajor<DH, kGRows>;
  using KT = KMajor<DH, kGTile>;
  __shared__ __attribute__((aligned(16))) float qs[DH * QT::kPitch];
  __shared__ __attribute__((aligned(16))) float ks[2][DH * KT::kPitch];
  __shared__ float red[2][4][kGRows];
  // block -> (half, then as the bf16 pass 1: query block, prompt, layer * Hq + head)
  int idx = blockIdx.x;
  const int half = idx & 1;
  idx >>= 1;
  const int lh = idx % (L * Hq);
  idx /= L * Hq;
  int b, qblk;
  if (blist) {
    const int2 e = blist[idx];
    if (e.x < 0) return;
    b = e.x;
    qblk = e.y;
  } else {
    b = idx % B;
    qblk = nqb_max - 1 - idx / B;
  }
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const int q_lo = 2 * kGRows * qblk + kGRows * half;  // first query of this workgroup
  if (q_lo >= N) return;
  const int l = lh / Hq, h = lh % Hq;
  const int g = h / (Hq / Hkv);
  const int tid = threadIdx.x, tk = tid >> 5, tq = tid & 31;
  const size_t qrow = size_t(Hq) * DH, krow = size_t(Hkv) * DH;
  const float* Qh = Q + (size_t(l) * n_tok + base) * qrow + size_t(h) * DH;
  const float* Kg = K + (size_t(l) * n_tok + base) * krow + size_t(g) * DH;

  {
    QT ql;
    ql.load(tid, [&](int r) { return Qh + size_t(min(q_lo + r, N - 1)) * qrow; });
    ql.store(tid, qs);
  }
  const int q_hi = min(N, q_lo + kGRows);  // end of the workgroup's queries
  const int n_kt = (q_hi - 1) / kGTile + 1;
  KT kl;
  kl.load(tid, [&](int r) { return Kg + size_t(min(r, N - 1)) * krow; });
  kl.store(tid, ks[0]);
  __syncthreads();

  const int q0 = q_lo + 4 * tq;  // the thread's first query
  float m[4], s[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    m[j] = -INFINITY;
    s[j] = 0.f;
  }
  for (int kt = 0; kt < n_kt; ++kt) {
    const bool more = kt + 1 < n_kt;
    if (more) kl.load(tid, [&](int r) { return Kg + size_t(min((kt + 1) * kGTile + r, N - 1)) * krow; });
    const int k0 = kt * kGTile;
    if (q0 < N && k0 + 4 * tk <= q0 + 3) {  // some key of the thread is visible to some query of it
      float sc[8][4];
      scores_8x4<DH, KT::kPitch, QT::kPitch>(ks[kt & 1], 4 * tk, qs, 4 * tq, sc);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int qi = q0 + j;
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int kj = k0 + (i < 4 ? 4 * tk + i : 32 + 4 * tk + i - 4);
          sc[i][j] = kj <= qi ? sc[i][j] * c2 : -INFINITY;  // keys after the query are masked
          mx = fmaxf(mx, sc[i][j]);
        }
        if (mx == -INFINITY) continue;  // none of the thread's keys is visible to this query
        const float mnew = fmaxf(m[j], mx);
        float sum = s[j] * fast_exp2(fmaxf(m[j] - mnew, kExp2Floor));
#pragma unroll
        for (int i = 0; i < 8; ++i) sum += fast_exp2(sc[i][j] - mnew);
        m[j] = mnew;
        s[j] = sum;
      }
    }
    if (more) kl.store(tid, ks[(kt + 1) & 1]);
    __syncthreads();
  }
  // the 8 threads of a query: tk's low bit within the wave (lane ^ 32), then the 4 waves in order
  const int wave = tid >> 6, lane = tid & 63;
#pragma unroll
  for (int j = 0; j < 4; ++j) lse_merge(m[j], s[j], __shfl_xor(m[j], 32, 64), __shfl_xor(s[j], 32, 64));
  if (lane < 32) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      red[0][wave][4 * tq + j] = m[j];
      red[1][wave][4 * tq + j] = s[j];
    }
  }
  __syncthreads();
  if (tid < kGRows && q_lo + tid < N) {
    float M = red[0][0][tid], S = red[1][0][tid];
    for (int w = 1; w < 4; ++w) lse_merge(M, S, red[0][w][tid], red[1][w][tid]);
    lse2[(size_t(l) * Hq + h) * n_tok + base + q_lo + tid] = M + fast_log2(S);
  }
}

template <int DH>
__global__ __launch_bounds__(kGThreads) void attn_colsum_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const int* __restrict__ cu, int B, int n_tok, int L,
    int Hq, int Hkv, float c2, const float* __restrict__ lse2, float lse_mul, int strict,
    const int2* __restrict__ blist, int n_blist, float* __restrict__ part) {
  using KT = KMajor<DH, kGRows>;
  using QT = KMajor<DH, kGTile>;
  __shared__ __attribute__((aligned(16))) float ks[DH * KT::kPitch];
  __shared__ __attribute__((aligned(16))) float qs[2][DH * QT::kPitch];
  __shared__ float ls[2][kGTile];
  __shared__ float red[4][kGRows];
  const int G = Hq / Hkv;
  // block -> (half, then as the bf16 pass 2: key block, prompt, layer * Hkv + KV head)
  int idx = blockIdx.x;
  const int half = idx & 1;
  idx >>= 1;
  const int lg = idx % (L * Hkv);
  idx /= L * Hkv;
  int b, kblk;
  if (blist) {
    const int2 e = blist[n_blist - 1 - idx];
    if (e.x < 0) return;
    b = e.x;
    kblk = e.y;
  } else {
    b = idx % B;
    kblk = idx / B;
  }
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const int k_lo = 2 * kGRows * kblk + kGRows * half;  // first key of this workgroup
  if (k_lo >= N) return;
  const int l = lg / Hkv, g = lg % Hkv;
  const int tid = threadIdx.x, tq = tid >> 5, tk = tid & 31;
  const size_t qrow = size_t(Hq) * DH, krow = size_t(Hkv) * DH;
  const float* Ql = Q + (size_t(l) * n_tok + base) * qrow;
  const float* Kg = K + (size_t(l) * n_tok + base) * krow + size_t(g) * DH;
  const float* Ll = lse2 + size_t(l) * Hq * n_tok + base;

  {
    KT kl;
    kl.load(tid, [&](int r) { return Kg + size_t(min(k_lo + r, N - 1)) * krow; });
    kl.store(tid, ks);
  }
  // tiles (64-query tile, head) from the workgroup's first key on, head fastest
  const int qt_first = k_lo / kGTile;
  const int n_tiles = ((N + kGTile - 1) / kGTile - qt_first) * G;
  QT ql;
  float lv = 0.f;
  auto fetch = [&](int t) {
    const int hh = g * G + t % G;
    const int i0 = (qt_first + t / G) * kGTile;
    ql.load(tid, [&](int r) { return Ql + size_t(min(i0 + r, N - 1)) * qrow + size_t(hh) * DH; });
    if (tid < kGTile) lv = i0 + tid < N ? Ll[size_t(hh) * n_tok + i0 + tid] * lse_mul : INFINITY;
  };
  auto put = [&](int buf) {
    ql.store(tid, qs[buf]);
    if (tid < kGTile) ls[buf][tid] = lv;
  };
  fetch(0);
  put(0);
  __syncthreads();

  const int kj0 = k_lo + 4 * tk;  // the thread's first key
  float cs[4] = {0.f, 0.f, 0.f, 0.f};
  for (int t = 0; t < n_tiles; ++t) {
    const bool more = t + 1 < n_tiles;
    if (more) fetch(t + 1);
    const int i0 = (qt_first + t / G) * kGTile;
    if (kj0 < N && i0 + 32 + 4 * tq + 3 >= kj0 + strict) {  // some query of the thread counts for some key of it
      float sc[8][4];
      scores_8x4<DH, QT::kPitch, KT::kPitch>(qs[t & 1], 4 * tq, ks, 4 * tk, sc);
      const float* lt = ls[t & 1];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = i < 4 ? 4 * tq + i : 32 + 4 * tq + i - 4;
        const int qi = i0 + r;
        const float lq = lt[r];  // +inf past N: weight 0
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p = fast_exp2(fmaf(sc[i][j], c2, -lq));
          cs[j] += qi >= kj0 + j + strict ? p : 0.f;
        }
      }
    }
    if (more) put((t + 1) & 1);
    __syncthreads();
  }
  // the 8 threads of a key: tq's low bit within the wave (lane ^ 32), then the 4 waves in order
  const int wave = tid >> 6, lane = tid & 63;
#pragma unroll
  for (int j = 0; j < 4; ++j) cs[j] += __shfl_xor(cs[j], 32, 64);
  if (lane < 32) {
#pragma unroll
    for (int j = 0; j < 4; ++j) red[wave][4 * tk + j] = cs[j];
  }
  __syncthreads();
  if (tid < kGRows && k_lo + tid < N) {
    const float v = ((red[0][tid] + red[1][tid]) + red[2][tid]) + red[3][tid];
    part[(size_t(l) * Hkv + g) * n_tok + base + k_lo + tid] = v;
  }
}

template <int DH>
static void launch_f32(const float* Q, const float* K, const int* cu, int B, int n_tok, int L, int Hq, int Hkv,
                       int nqb, float c2, const int2* blist, size_t n_rows, int n_bound, bool run_lse, float* lse2,
                       float lse_mul, int strict, float* part, hipStream_t s) {
  static_assert(2 * kGRows == 256, "two workgroups per 256-row block");
  if (run_lse)
    attn_lse_f32_kernel<DH><<<dim3(2 * n_rows * L * Hq), dim3(kGThreads), 0, s>>>(Q, K, cu, B, n_tok, L, Hq, Hkv,
                                                                                   nqb, c2, blist, lse2);
  attn_colsum_f32_kernel<DH><<<dim3(2 * n_rows * L * Hkv), dim3(kGThreads), 0, s>>>(
      Q, K, cu, B, n_tok, L, Hq, Hkv, c2, lse2, lse_mul, strict, blist, n_bound, part);
}

void launch_importance_f32(int dh, const float* Q, const float* K, const int* cu, int B, int n_tok, int L, int Hq,
                           int Hkv, int nqb, float c2, const int2* blist, size_t n_rows, int n_bound, bool run_lse,
                           float* lse2, float lse_mul, int strict, float* part, hipStream_t s) {
  switch (dh) {
    case 32:
      launch_f32<32>(Q, K, cu, B, n_tok, L, Hq, Hkv, nqb, c2, blist, n_rows, n_bound, run_lse, lse2, lse_mul, strict,
                     part, s);
      break;
    case 64:
      launch_f32<64>(Q, K, cu, B, n_tok, L, Hq, Hkv, nqb, c2, blist, n_rows, n_bound, run_lse, lse2, lse_mul, strict,
                     part, s);
      break;
    default:
      launch_f32<128>(Q, K, cu, B, n_tok, L, Hq, Hkv, nqb, c2, blist, n_rows, n_bound, run_lse, lse2, lse_mul,
                      strict, part, s);
      break;
  }
}

}  // namespace detail
}  // namespace estp
