// Attention importance (Eq. 1, Section 4.1) for fp32 queries and keys, with
// fp32 arithmetic throughout: the same two passes, grids and intermediate
// layouts as the bf16 matrix-core kernels, as VALU dot products.
//
// Pass 1 (attn_lse_f32_kernel): one workgroup per (256-query block, layer,
// query head); thread i keeps query i in registers and streams the prompt's
// keys through a double-buffered LDS tile of 32 keys (every thread reads the
// same key row at once: LDS broadcast).  Per tile the thread forms its 32
// scores, masks the keys after its query and folds them into an exact online
// log-sum-exp in base 2: lse2 = log2 sum_j 2^(c s_ij), c = scale * log2 e.
//
// Pass 2 (attn_colsum_f32_kernel): one workgroup per (256-key block, layer,
// KV head); thread j keeps key j in registers and streams every later
// 32-query tile of each query head of the group, with the tile's row lse2,
// summing 2^(c s_ij - lse2_i) over the queries i >= j (i > j when the
// diagonal is left out) into its column mass.  attn_reduce_kernel then
// divides by N * Hq as for the bf16 path.  No atomics: bitwise reproducible.
#include "estp_common.h"
#include "f32_paths.h"

namespace estp {
namespace detail {
namespace {

constexpr int kGThreads = 256;  // rows (queries or keys) per workgroup: the 256-row blocks of the bf16 path
constexpr int kGTile = 32;      // streamed keys (pass 1) or queries (pass 2) per LDS tile

// Loads of one 32-row tile of DH floats: each thread moves kGTile * DH / 4 / 256 float4.
template <int DH>
struct TileLoad {
  static constexpr int kPerThread = kGTile * DH / 4 / kGThreads;
  static_assert(kPerThread >= 1 && kGTile * DH / 4 % kGThreads == 0, "tile load pattern");
  float4 v[kPerThread];
  // row r of the tile comes from rowptr(r) (a clamped, valid row)
  template <class RowPtr>
  __device__ __forceinline__ void load(int tid, RowPtr rowptr) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int idx = tid + kGThreads * i;
      v[i] = *reinterpret_cast<const float4*>(rowptr(idx / (DH / 4)) + 4 * (idx % (DH / 4)));
    }
  }
  __device__ __forceinline__ void store(int tid, float (*tile)[DH]) const {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int idx = tid + kGThreads * i;
      *reinterpret_cast<float4*>(&tile[idx / (DH / 4)][4 * (idx % (DH / 4))]) = v[i];
    }
  }
};

// 32 dot products of the thread's register row with the rows of an LDS tile
template <int DH>
__device__ __forceinline__ void tile_dots(const float (&x)[DH], const float (*tile)[DH], float (&dot)[kGTile]) {
#pragma unroll
  for (int r = 0; r < kGTile; ++r) dot[r] = 0.f;
#pragma unroll
  for (int c = 0; c < DH; c += 4) {
#pragma unroll
    for (int r = 0; r < kGTile; ++r) {
      const float4 y = *reinterpret_cast<const float4*>(&tile[r][c]);
      dot[r] = fmaf(x[c], y.x, dot[r]);
      dot[r] = fmaf(x[c + 1], y.y, dot[r]);
      dot[r] = fmaf(x[c + 2], y.z, dot[r]);
      dot[r] = fmaf(x[c + 3], y.w, dot[r]);
    }
  }
}

template <int DH>
__device__ __forceinline__ void load_row(const float* p, float (&x)[DH]) {
#pragma unroll
  for (int c = 0; c < DH; c += 4) {
    const float4 v = *reinterpret_cast<const float4*>(p + c);
    x[c] = v.x;
    x[c + 1] = v.y;
    x[c + 2] = v.z;
    x[c + 3] = v.w;
  }
}

}  // namespace

template <int DH>
__global__ __launch_bounds__(kGThreads) void attn_lse_f32_kernel(const float* __restrict__ Q,
                                                                 const float* __restrict__ K,
                                                                 const int* __restrict__ cu, int B, int n_tok, int L,
                                                                 int Hq, int Hkv, int nqb_max, float c2,
                                                                 const int2* __restrict__ blist,
                                                                 float* __restrict__ lse2) {
  __shared__ __attribute__((aligned(16))) float ktile[2][kGTile][DH];
  // block -> (query block, prompt, layer * Hq + head), as the bf16 pass 1
  int idx = blockIdx.x;
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
  if (qblk * kGThreads >= N) return;
  const int l = lh / Hq, h = lh % Hq;
  const int g = h / (Hq / Hkv);
  const int tid = threadIdx.x;
  const size_t qrow = size_t(Hq) * DH, krow = size_t(Hkv) * DH;
  const float* Qh = Q + (size_t(l) * n_tok + base) * qrow + size_t(h) * DH;
  const float* Kg = K + (size_t(l) * n_tok + base) * krow + size_t(g) * DH;

  const int qi = qblk * kGThreads + tid;
  float q[DH];
  load_row<DH>(Qh + size_t(min(qi, N - 1)) * qrow, q);
  const int q_hi = min(N, qblk * kGThreads + kGThreads);  // end of the block's queries
  const int n_kt = (q_hi - 1) / kGTile + 1;                // key tiles the block needs

  TileLoad<DH> ld;
  auto fetch = [&](int kt) {
    ld.load(tid, [&](int r) { return Kg + size_t(min(kt * kGTile + r, N - 1)) * krow; });
  };
  fetch(0);
  ld.store(tid, ktile[0]);
  __syncthreads();
  float m = -INFINITY, s = 0.f;  // running max and sum of 2^(c s - m) of this thread's query
  for (int kt = 0; kt < n_kt; ++kt) {
    const bool more = kt + 1 < n_kt;
    if (more) fetch(kt + 1);
    const int k0 = kt * kGTile;
    if (qi < N && k0 <= qi) {
      float dot[kGTile];
      tile_dots<DH>(q, ktile[kt & 1], dot);
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < kGTile; ++r) {
        dot[r] = k0 + r <= qi ? dot[r] * c2 : -INFINITY;  // keys after the query are masked
        mx = fmaxf(mx, dot[r]);
      }
      const float mnew = fmaxf(m, mx);  // finite: key k0 <= qi is always visible
      float sum = s * fast_exp2(fmaxf(m - mnew, kExp2Floor));
#pragma unroll
      for (int r = 0; r < kGTile; ++r) sum += fast_exp2(dot[r] - mnew);
      m = mnew;
      s = sum;
    }
    if (more) ld.store(tid, ktile[(kt + 1) & 1]);
    __syncthreads();
  }
  if (qi < N) lse2[(size_t(l) * Hq + h) * n_tok + base + qi] = m + fast_log2(s);
}

template <int DH>
__global__ __launch_bounds__(kGThreads) void attn_colsum_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const int* __restrict__ cu, int B, int n_tok, int L,
    int Hq, int Hkv, float c2, const float* __restrict__ lse2, float lse_mul, int strict,
    const int2* __restrict__ blist, int n_blist, float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) float qtile[2][kGTile][DH];
  __shared__ float ltile[2][kGTile];
  const int G = Hq / Hkv;
  // block -> (key block, prompt, layer * Hkv + kv head), as the bf16 pass 2
  int idx = blockIdx.x;
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
  if (kblk * kGThreads >= N) return;
  const int l = lg / Hkv, g = lg % Hkv;
  const int tid = threadIdx.x;
  const size_t qrow = size_t(Hq) * DH, krow = size_t(Hkv) * DH;
  const float* Ql = Q + (size_t(l) * n_tok + base) * qrow;
  const float* Kg = K + (size_t(l) * n_tok + base) * krow + size_t(g) * DH;
  const float* Ll = lse2 + size_t(l) * Hq * n_tok + base;

  const int j = kblk * kGThreads + tid;  // this thread's key
  float kr[DH];
  load_row<DH>(Kg + size_t(min(j, N - 1)) * krow, kr);

  // tiles (query tile qt, head) from the block's first key on, head fastest
  const int qt_first = kblk * kGThreads / kGTile;
  const int n_tiles = ((N + kGTile - 1) / kGTile - qt_first) * G;
  TileLoad<DH> ld;
  float lv = 0.f;
  auto fetch = [&](int t) {
    const int hh = g * G + t % G;
    const int i0 = (qt_first + t / G) * kGTile;
    ld.load(tid, [&](int r) { return Ql + size_t(min(i0 + r, N - 1)) * qrow + size_t(hh) * DH; });
    if (tid < kGTile) lv = i0 + tid < N ? Ll[size_t(hh) * n_tok + i0 + tid] * lse_mul : INFINITY;
  };
  auto put = [&](int buf) {
    ld.store(tid, qtile[buf]);
    if (tid < kGTile) ltile[buf][tid] = lv;
  };
  fetch(0);
  put(0);
  __syncthreads();
  float cs = 0.f;
  for (int t = 0; t < n_tiles; ++t) {
    const bool more = t + 1 < n_tiles;
    if (more) fetch(t + 1);
    const int i0 = (qt_first + t / G) * kGTile;
    if (j < N && i0 + kGTile - 1 >= j + strict) {  // some query of the tile counts for this key
      float dot[kGTile];
      tile_dots<DH>(kr, qtile[t & 1], dot);
#pragma unroll
      for (int r = 0; r < kGTile; ++r) {
        const float p = fast_exp2(fmaf(dot[r], c2, -ltile[t & 1][r]));  // rows past N carry lse +inf: 0
        cs += i0 + r >= j + strict ? p : 0.f;
      }
    }
    if (more) put((t + 1) & 1);
    __syncthreads();
  }
  if (j < N) part[(size_t(l) * Hkv + g) * n_tok + base + j] = cs;
}

template <int DH>
static void launch_f32(const float* Q, const float* K, const int* cu, int B, int n_tok, int L, int Hq, int Hkv,
                       int nqb, float c2, const int2* blist, size_t n_rows, int n_bound, bool run_lse, float* lse2,
                       float lse_mul, int strict, float* part, hipStream_t s) {
  if (run_lse)
    attn_lse_f32_kernel<DH><<<dim3(n_rows * L * Hq), dim3(kGThreads), 0, s>>>(Q, K, cu, B, n_tok, L, Hq, Hkv, nqb,
                                                                               c2, blist, lse2);
  attn_colsum_f32_kernel<DH><<<dim3(n_rows * L * Hkv), dim3(kGThreads), 0, s>>>(
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
