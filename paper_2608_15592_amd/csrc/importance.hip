// Attention importance, Eq. 1 (Section 4.1):
//   S_j = sum_l (1/N) sum_{i >= j} (1/Hq) sum_h A^{l,h}_{ij}
// with A the causal softmax of scale * q_i . k_j inside each prompt, without
// ever forming the N x N attention.
//
// Pass 1 (attn_lse_kernel): one workgroup per (layer, query head, prompt,
// 256-query block); each of its 4 waves keeps 64 queries as matrix-core B
// fragments in registers and streams the prompt's 64-key blocks through a
// double-buffered LDS tile (global -> LDS transfers, chunk-swizzled).  Scores
// are formed as S^T = K Q^T (keys on the MFMA "M" side), so a lane owns one
// query column and 32 key rows of each block: the online max / sum over keys
// is per lane.  Output: lse2 = log2 sum_j 2^(c s_ij), c = scale * log2 e.
//
// Pass 2 (attn_colsum_kernel): one workgroup per (layer, KV head, prompt,
// 256-key block); each wave keeps 64 keys as B fragments in registers and
// streams, through LDS, every later 64-query block of every query head that
// shares the KV head (grouped-query reuse: the keys are read once).  When that
// grid is small, the group's query heads are split over a few workgroups per
// key block, each writing its own row of column masses.  Scores
// are formed as S = Q K^T, so a lane owns one key column and 16 query rows of
// each 32 x 32 block; 2^(c s - lse2) is summed per lane into column sums.
// Partial column masses per (layer, KV head) are reduced in a fixed order by
// attn_reduce_kernel, which divides by N * Hq.  No atomics: results are
// bitwise reproducible.  Both passes are register-bounded to three waves per
// SIMD (168 VGPRs, no spills) so that one wave's exponentials overlap the
// others' matrix-core work.
#include <algorithm>

#include "estp_common.h"
#include "f32_paths.h"

namespace estp {
namespace detail {

// 32-wide column blocks a wave keeps resident.  One block per wave (eight waves of 32 rows, four
// waves per SIMD) was measured slower on MI355X than two: 5.80 against 5.50 ms per call on 32 x
// 2048 tokens, 32/8 heads of 128, 4 layers (twice the LDS fragment reads per MFMA).
constexpr int kNC = 2;
constexpr int kWaves = 8 / kNC;       // waves per 256-row block
constexpr int kThreads = 64 * kWaves;
constexpr int kMinBlocks = 3;         // workgroups per CU the register budget is sized for
constexpr int kQPerWave = 32 * kNC;  // queries per wave in pass 1
constexpr int kQBlock = kWaves * kQPerWave;
constexpr int kKPerWave = 32 * kNC;  // keys per wave in pass 2
constexpr int kKBlock = kWaves * kKPerWave;
constexpr int kKTile = 64;     // keys per streamed tile in pass 1
constexpr int kQTile = 64;     // queries per streamed tile in pass 2 (two 32-query row blocks in turn)
static_assert(kKBlock % kQTile == 0 && kQTile % 32 == 0, "pass-2 tiles must tile a key block");

// Upper bound on the live 256-row blocks: sum_b ceil(N_b / 256) <= n_tok / 256 + B.
inline size_t block_bound(int64_t n_tok, int32_t B, int32_t max_seqlen) {
  const size_t nblk = (size_t(max_seqlen) + kQBlock - 1) / kQBlock;
  const size_t a = size_t(B) * nblk, c = size_t(n_tok) / kQBlock + size_t(B);
  return a < c ? a : c;
}

// Grids sized by the longest prompt are mostly workgroups that exit at once when the lengths
// vary widely; then both passes run over the list of live blocks instead.
inline bool use_block_list(int64_t n_tok, int32_t B, int32_t max_seqlen) {
  const size_t nqb = (size_t(max_seqlen) + kQBlock - 1) / kQBlock;
  return block_bound(n_tok, B, max_seqlen) * 4 < size_t(B) * nqb * 3;
}

// 256-row block entries of either grid (rows of the pass grids)
inline size_t block_rows(int64_t n_tok, int32_t B, int32_t max_seqlen) {
  const size_t nqb = (size_t(max_seqlen) + kQBlock - 1) / kQBlock;
  return use_block_list(n_tok, B, max_seqlen) ? block_bound(n_tok, B, max_seqlen) : size_t(B) * nqb;
}

// Query heads of one KV group are split over `nsplit` pass-2 workgroups when the grid would
// otherwise be small: the smallest divisor of G = Hq / Hkv that gives at least four workgroups per
// compute unit (else G, one head each).  The fp32 kernels keep one workgroup per group.
inline int colsum_split(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t L, int32_t Hq, int32_t Hkv, bool f32) {
  if (f32) return 1;
  const int G = Hq / Hkv;
  const int n_cu = std::max(1, current_device_cu_count());
  const size_t base = block_rows(n_tok, B, max_seqlen) * size_t(L) * size_t(Hkv);
  for (int d = 1; d < G; ++d)
    if (G % d == 0 && base * size_t(d) >= size_t(4) * n_cu) return d;
  return G;
}

// Rows of DH bf16 staged in LDS: 16-byte chunks XOR-swizzled so that 16
// consecutive rows read at one logical chunk hit 16 distinct bank groups.
template <int DH>
struct RowTile {
  static constexpr int kRowBytes = DH * 2;
  static constexpr int kChunks = kRowBytes / 16;
  static constexpr int kRowsPerInst = 64 / kChunks;  // rows one wave-wide 16-byte transfer fills
  static constexpr int kRowsPerWindow = kRowBytes >= 256 ? 1 : 256 / kRowBytes;
  __device__ static __forceinline__ int swz(int row, int chunk) {
    return chunk ^ ((row / kRowsPerWindow) & (kChunks - 1));
  }
  // byte offset of the fragment (row, logical chunk)
  __device__ static __forceinline__ int off(int row, int chunk) { return row * kRowBytes + swz(row, chunk) * 16; }
};

// Wave-cooperative staging of `rows` rows into LDS at `dst`; tile row r comes
// from `src_row(r)`.  Waves take groups of kRowsPerInst rows round-robin.
template <int DH, typename RowPtr>
__device__ __forceinline__ void stage_rows(char* dst, int rows, int wave, int nwaves, int lane, RowPtr src_row) {
  using T = RowTile<DH>;
  for (int r0 = wave * T::kRowsPerInst; r0 < rows; r0 += nwaves * T::kRowsPerInst) {
    const int r = r0 + lane / T::kChunks;
    const int chunk = T::swz(r, lane % T::kChunks);
    lds_dma16(reinterpret_cast<const char*>(src_row(r)) + chunk * 16, dst + r0 * T::kRowBytes);
  }
}

// ---------------------------------------------------------------- pass 1
template <int DH>
__global__ __launch_bounds__(kThreads, kMinBlocks) void attn_lse_kernel(const uint16_t* __restrict__ Q,
                                                            const uint16_t* __restrict__ K,
                                                            const int* __restrict__ cu, int B, int n_tok,
                                                            int L, int Hq, int Hkv, int nqb_max, float c2,
                                                            const int2* __restrict__ blist, int xcd_groups,
                                                            float* __restrict__ lse2) {
  constexpr int KS = DH / 16;
  using T = RowTile<DH>;
  constexpr int kTileBytes = kKTile * T::kRowBytes;
  __shared__ __attribute__((aligned(16))) char ktile[2][kTileBytes];

  // block -> (query block, prompt, layer * Hq + head); largest query blocks first
  // or, when many prompts are much shorter than the longest, the entry of the list of live
  // 256-row blocks (already heaviest first)
  int idx = blockIdx.x;
  int lh;
  if (xcd_groups) {
    // Workgroups are dealt to the 8 XCDs in turn (block id mod 8), each with its own L2. The G
    // query heads of one KV group read the same key tiles in the same order, so ids 8s + x for
    // s = G u', ..., G u' + G - 1 (one XCD, back to back) take the G heads of unit u = 8 u' + x,
    // where units (block row, layer, KV head) keep the order of the plain grid.
    const int G = Hq / Hkv;
    const int x = idx & 7, sx = idx >> 3;
    const int u = (sx / G) * 8 + x;
    lh = (u % (L * Hkv)) * G + sx % G;
    idx = u / (L * Hkv);
  } else {
    lh = idx % (L * Hq);
    idx /= L * Hq;
  }
  int b, qblk;
  if (blist) {
    const int2 e = blist[idx];
    if (e.x < 0) return;  // past the live blocks
    b = e.x;
    qblk = e.y;
  } else {
    b = idx % B;
    qblk = nqb_max - 1 - idx / B;
  }
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  if (qblk * kQBlock >= N) return;
  const int l = lh / Hq, h = lh % Hq;
  const int g = h / (Hq / Hkv);

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 31;   // query column of this lane in a 32 x 32 block
  const int half = lane >> 5;  // 8-wide k half of the fragment / row quad of the output
  const size_t qrow = size_t(Hq) * DH, krow = size_t(Hkv) * DH;
  const uint16_t* Qh = Q + size_t(l) * n_tok * qrow + size_t(base) * qrow + size_t(h) * DH;
  const uint16_t* Kg = K + size_t(l) * n_tok * krow + size_t(base) * krow + size_t(g) * DH;

  const int q0 = qblk * kQBlock + wave * kQPerWave;  // this wave's first query
  auto qcb = [&](int cb) { return q0 + 32 * cb; };  // first query of column block cb
  const int q_hi = min(N, qblk * kQBlock + kQBlock);  // end of the block's queries
  const int n_kt = (q_hi - 1) / kKTile + 1;           // key tiles the block needs

  // queries as B fragments: column cb*32 + col, k = 16 ks + 8 half
  bf16x8_t bq[kNC][KS];
#pragma unroll
  for (int cb = 0; cb < kNC; ++cb) {
    const int qi = min(qcb(cb) + col, N - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      bq[cb][ks] = *reinterpret_cast<const bf16x8_t*>(Qh + size_t(qi) * qrow + ks * 16 + half * 8);
  }
  float m[kNC], s[kNC];
#pragma unroll
  for (int cb = 0; cb < kNC; ++cb) {
    m[cb] = -INFINITY;
    s[cb] = 0.f;
  }

  auto stage = [&](int kt, int buf) {
    stage_rows<DH>(ktile[buf], kKTile, wave, kWaves, lane,
                   [&](int r) { return Kg + size_t(min(kt * kKTile + r, N - 1)) * krow; });
  };
  stage(0, 0);
  for (int kt = 0; kt < n_kt; ++kt) {
    wait_vm<0>();
    lds_barrier();  // tile kt visible; every wave is done with buffer (kt + 1) & 1
    if (kt + 1 < n_kt) stage(kt + 1, (kt + 1) & 1);
    const int k0 = kt * kKTile;
    if (k0 > qcb(kNC - 1) + 31 || qcb(0) >= N) continue;  // whole tile after this wave's queries
    const char* kb = ktile[kt & 1];
    f32x16_t acc[2][kNC];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int cb = 0; cb < kNC; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[rb][cb][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(kb + T::off(rb * 32 + col, ks * 2 + half));
#pragma unroll
        for (int cb = 0; cb < kNC; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[cb][ks], acc[rb][cb], 0, 0, 0);
      }
    }
    // acc[rb][cb][r]: key k0 + rb*32 + 8*(r/4) + 4*half + r%4, query q0 + cb*32 + col
    // Running state per query column: reference m (base-2 units) and
    // s = sum 2^(c2 s_ij - m).  After the first tile m is rebased to the
    // running log-sum-exp (s = 1), so later tiles fold with one FMA, one exp2
    // and one add per score and no max pass; a tile that would push s past
    // 2^64 (or a lane with no reference yet) is refolded exactly with its max.
#pragma unroll
    for (int cb = 0; cb < kNC; ++cb) {
      if (k0 > qcb(cb) + 31 || qcb(cb) >= N) continue;  // every key after every query: nothing to fold
      const bool diag = k0 + kKTile - 1 > qcb(cb);
      if (diag) {
        // key k0 + rb*32 + 4*half + off(r) lies after query qi iff off(r) > qi - k0 - rb*32 - 4*half,
        // with off(r) = 8*(r/4) + r%4 a constant: one compare per score, no index arithmetic
        const int t0 = qcb(cb) + col - k0 - 4 * half;
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (8 * (r >> 2) + (r & 3) > t0 - rb * 32) acc[rb][cb][r] = -INFINITY;
      }
      // four partial sums in a fixed order: no serial chain through one accumulator
      float s4[4] = {s[cb], 0.f, 0.f, 0.f};
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s4[r & 3] += fast_exp2(fmaf(acc[rb][cb][r], c2, -m[cb]));
      float sum = (s4[0] + s4[1]) + (s4[2] + s4[3]);
      if (!(sum <= 0x1p64f)) {  // overflow, NaN from m = -inf, or far above the reference
        float mx = acc[0][cb][0];
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, acc[rb][cb][r]);
        const float mnew = fmaxf(m[cb], mx * c2);
        sum = s[cb] * fast_exp2(fmaxf(m[cb] - mnew, kExp2Floor));
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int r = 0; r < 16; ++r) sum += fast_exp2(fmaf(acc[rb][cb][r], c2, -mnew));
        // nothing seen yet in this lane (all keys masked): fmaf(-inf, c2, inf) is NaN, keep the empty state
        sum = (mnew == -INFINITY) ? 0.f : sum;
        m[cb] = mnew;
      }
      // rebase to the running log-sum-exp (s >= 1 whenever anything was seen)
      if (sum > 0.f) {
        m[cb] += fast_log2(sum);
        sum = 1.f;
      }
      s[cb] = sum;
    }
  }
  // lanes col and col + 32 hold the two row quads of the same query column
#pragma unroll
  for (int cb = 0; cb < kNC; ++cb) {
    const float mo = __shfl_xor(m[cb], 32, 64);
    const float so = __shfl_xor(s[cb], 32, 64);
    const float M = fmaxf(m[cb], mo);
    const float tot = s[cb] * fast_exp2(fmaxf(m[cb] - M, kExp2Floor)) + so * fast_exp2(fmaxf(mo - M, kExp2Floor));
    const int qi = qcb(cb) + col;
    if (half == 0 && qi < N) lse2[(size_t(l) * Hq + h) * n_tok + base + qi] = M + fast_log2(tot);
  }
}

// ---------------------------------------------------------------- pass 2
template <int DH>
__global__ __launch_bounds__(kThreads, kMinBlocks) void attn_colsum_kernel(const uint16_t* __restrict__ Q,
                                                               const uint16_t* __restrict__ K,
                                                               const int* __restrict__ cu, int B, int n_tok,
                                                               int L, int Hq, int Hkv, float c2,
                                                               const float* __restrict__ lse2, float lse_mul,
                                                               int strict, const int2* __restrict__ blist,
                                                               int n_blist, int nsplit, float* __restrict__ part) {
  constexpr int KS = DH / 16;
  using T = RowTile<DH>;
  constexpr int kTileBytes = kQTile * T::kRowBytes;
  __shared__ __attribute__((aligned(16))) char qtile[2][kTileBytes];
  __shared__ __attribute__((aligned(16))) float ltile[2][kQTile];

  const int G = Hq / Hkv;
  const int hpw = G / nsplit;  // query heads this workgroup walks: hs * hpw .. of the group
  // block -> (key block, prompt, (layer * Hkv + kv head) * nsplit + head share); key block 0 (the
  // most work) first, or the list of live 256-row blocks walked from its end (lightest first
  // there, so heaviest first here; the padding entries past the live ones come first and exit)
  int idx = blockIdx.x;
  const int lgs = idx % (L * Hkv * nsplit);
  idx /= L * Hkv * nsplit;
  const int lg = lgs / nsplit, hs = lgs % nsplit;
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
  if (kblk * kKBlock >= N) return;
  const int l = lg / Hkv, g = lg % Hkv;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 31;   // key column of this lane in a 32 x 32 block
  const int half = lane >> 5;
  const size_t qrow = size_t(Hq) * DH, krow = size_t(Hkv) * DH;
  const uint16_t* Ql = Q + size_t(l) * n_tok * qrow + size_t(base) * qrow;
  const uint16_t* Kg = K + size_t(l) * n_tok * krow + size_t(base) * krow + size_t(g) * DH;
  const float* Ll = lse2 + size_t(l) * Hq * n_tok + base;

  const int k0 = kblk * kKBlock + wave * kKPerWave;  // this wave's first key
  auto kcb = [&](int cb) { return k0 + 32 * cb; };  // first key of column block cb
  // keys as B fragments, resident for the whole walk
  bf16x8_t bk[kNC][KS];
#pragma unroll
  for (int cb = 0; cb < kNC; ++cb) {
    const int kj = min(kcb(cb) + col, N - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      bk[cb][ks] = *reinterpret_cast<const bf16x8_t*>(Kg + size_t(kj) * krow + ks * 16 + half * 8);
  }
  float csum[kNC];
#pragma unroll
  for (int cb = 0; cb < kNC; ++cb) csum[cb] = 0.f;

  // tiles: (query block qb, head) for qb from the block's first key on; head fastest
  const int qb_first = kblk * (kKBlock / kQTile);
  const int n_qb = (N + kQTile - 1) / kQTile - qb_first;
  const int n_tiles = n_qb * hpw;
  const int h0 = g * G + hs * hpw;  // first query head of this workgroup's share
  auto stage = [&](int t, int buf) {
    const int hh = h0 + t % hpw;
    const int qb = qb_first + t / hpw;
    stage_rows<DH>(qtile[buf], kQTile, wave, kWaves, lane,
                   [&](int r) { return Ql + size_t(min(qb * kQTile + r, N - 1)) * qrow + size_t(hh) * DH; });
  };
  auto lse_load = [&](int t) {  // lanes below kQTile of wave 0 fetch the tile's row LSEs
    const int hh = h0 + t % hpw;
    const int i = (qb_first + t / hpw) * kQTile + lane;
    return (lane < kQTile && i < N) ? Ll[size_t(hh) * n_tok + i] * lse_mul : INFINITY;  // rows past N weigh 0
  };

  stage(0, 0);
  float lv = (wave == 0) ? lse_load(0) : 0.f;
  if (wave == 0 && lane < kQTile) ltile[0][lane] = lv;
  for (int t = 0; t < n_tiles; ++t) {
    wait_vm<0>();
    lds_barrier();  // tile t (queries and LSEs) visible; every wave is done with buffer (t + 1) & 1
    const bool more = t + 1 < n_tiles;
    if (more) {
      stage(t + 1, (t + 1) & 1);
      if (wave == 0) lv = lse_load(t + 1);
    }
    const int qb = qb_first + t / hpw;
    const int i0 = qb * kQTile;
    if (i0 + kQTile - 1 >= kcb(0) && kcb(0) < N) {  // some query of the tile sees some key of this wave
      const char* qt = qtile[t & 1];
      const float4* lp = reinterpret_cast<const float4*>(ltile[t & 1]);
      // tiles holding some query i <= (or, strict, ==) a key of a column block need the mask
      // The tile's 32-query row blocks go one after another through the same
      // accumulators: the tile, and so the barrier, is twice as long as one
      // 32 x 64 block of scores without a second set of registers.
#pragma unroll
      for (int rb = 0; rb < kQTile / 32; ++rb) {
        f32x16_t acc[kNC];
#pragma unroll
        for (int cb = 0; cb < kNC; ++cb)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[cb][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(qt + T::off(rb * 32 + col, ks * 2 + half));
#pragma unroll
          for (int cb = 0; cb < kNC; ++cb)
            acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bk[cb][ks], acc[cb], 0, 0, 0);
        }
        // acc[cb][r]: query i0 + rb*32 + 8*(r/4) + 4*half + r%4, key k0 + cb*32 + col
        float lr[16];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float4 v = lp[rb * 8 + 2 * q4 + half];  // rows rb*32 + 8 q4 + 4 half .. + 3
          lr[4 * q4] = v.x;
          lr[4 * q4 + 1] = v.y;
          lr[4 * q4 + 2] = v.z;
          lr[4 * q4 + 3] = v.w;
        }
#pragma unroll
        for (int cb = 0; cb < kNC; ++cb) {
          // every query of the row block before every key of the column block (or past the prompt)
          if (i0 + rb * 32 + 31 < kcb(cb) + strict || kcb(cb) >= N) continue;
          const bool diag = i0 < kcb(cb) + 31 + strict;
          float cs = 0.f;
          if (diag) {
            // query i = i0 + rb*32 + 4*half + off(r) counts for key j iff j < i + 1 - strict, i.e.
            // off(r) > j - i0 - rb*32 - 4*half - 1 + strict with off(r) = 8*(r/4) + r%4 a constant
            const int t = kcb(cb) + col - i0 - rb * 32 - 4 * half - 1 + strict;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float p = fast_exp2(fmaf(acc[cb][r], c2, -lr[r]));
              cs += (8 * (r >> 2) + (r & 3) > t) ? p : 0.f;
            }
          } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) cs += fast_exp2(fmaf(acc[cb][r], c2, -lr[r]));
          }
          csum[cb] += cs;
        }
      }
    }
    if (more && wave == 0 && lane < kQTile) ltile[(t + 1) & 1][lane] = lv;
  }
  // the two row quads (lane, lane + 32) of each key column
#pragma unroll
  for (int cb = 0; cb < kNC; ++cb) {
    csum[cb] += __shfl_xor(csum[cb], 32, 64);
    const int j = kcb(cb) + col;
    if (half == 0 && j < N) part[((size_t(l) * Hkv + g) * nsplit + hs) * n_tok + base + j] = csum[cb];
  }
}

// List of the live 256-row blocks, (prompt, block) with the block index descending and the
// prompt ascending within a block index, then (-1, 0) up to n_bound.  One workgroup: per block
// index, a scan over the prompts places the prompts that reach it.  Writes stop at n_bound, so a
// max_seqlen below the longest prompt (invalid input) stays inside the workspace.
__global__ __launch_bounds__(1024) void block_list_kernel(const int* __restrict__ cu, int B, int nblk, int n_bound,
                                                          int2* __restrict__ list) {
  __shared__ int wsum[16];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  int base = 0;
  for (int k = nblk - 1; k >= 0; --k) {
    for (int b0 = 0; b0 < B; b0 += 1024) {
      const int b = b0 + t;
      const int flag = (b < B && cu[b + 1] - cu[b] > k * kQBlock) ? 1 : 0;
      int x = flag;  // inclusive scan within the wave, then over the 16 wave totals
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
      const int pos = base + before + x - flag;
      if (flag && pos < n_bound) list[pos] = make_int2(b, k);
      base += total;
      __syncthreads();  // wsum is rewritten by the next round
    }
  }
  for (int i = base + t; i < n_bound; i += 1024) list[i] = make_int2(-1, 0);
}

constexpr int kMaxWeightedLayers = 64;
struct LayerWeights {
  float w[kMaxWeightedLayers];
};

// S_j = (sum over layers l and the column-mass rows of each layer (KV heads, or shares of their
// query heads) of w_l times the column masses) / (N * Hq); `Hkv` here counts those rows per layer
__global__ __launch_bounds__(256) void attn_reduce_kernel(const float* __restrict__ part, const int* __restrict__ cu,
                                                          int n_tok, int L, int Hkv, int Hq, int weighted,
                                                          LayerWeights lw, float* __restrict__ S) {
  const int b = blockIdx.y;
  const int base = cu[b];
  const int N = cu[b + 1] - base;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= N) return;
  float v = 0.f;
  for (int l = 0; l < L; ++l) {
    float vl = 0.f;
    for (int g = 0; g < Hkv; ++g) vl += part[(size_t(l) * Hkv + g) * n_tok + base + j];
    v = weighted ? fmaf(lw.w[l], vl, v) : v + vl;
  }
  S[base + j] = v / (float(N) * float(Hq));
}

// The definition block_list_kernel follows, on the host (debug checks): (prompt, block) for
// every block index from the last down, prompts ascending within it, then (-1, 0) fill.
std::vector<int2> block_list_on_host(const std::vector<int>& cu, int B, int nblk, size_t n_bound) {
  std::vector<int2> out;
  for (int k = nblk - 1; k >= 0; --k)
    for (int b = 0; b < B; ++b)
      if (cu[b + 1] - cu[b] > k * kQBlock) out.push_back(make_int2(b, k));
  out.resize(std::max(out.size(), n_bound), make_int2(-1, 0));
  out.resize(n_bound);
  return out;
}

template <int DH>
int launch(const char* fn, const void* Qv, const void* Kv, bool f32, const int* cu, int B, int max_seqlen, int n_tok,
           int L, int Hq, int Hkv, float scale, const float* lse_in, int strict, const float* layer_weights, float* S,
           float* lse2, float* part, int2* blist, hipStream_t s) {
  const int nsplit = colsum_split(n_tok, B, max_seqlen, L, Hq, Hkv, f32);  // part holds L * Hkv * nsplit rows
  static_assert(kQBlock == kKBlock, "the two passes share one list of 256-row blocks");
  const float c2 = scale * kLog2e;
  const int nqb = (max_seqlen + kQBlock - 1) / kQBlock;
  const size_t n_bound = block_bound(n_tok, B, max_seqlen);
  const bool use_list = use_block_list(n_tok, B, max_seqlen);
  if (debug_checks_enabled()) {  // cu_seqlens before any kernel reads it
    std::vector<int> cu_h;
    const int st = debug_check_cu(fn, cu, B, n_tok, max_seqlen, s, &cu_h);
    if (st != ESTP_OK) return st;
    if (use_list) {
      block_list_kernel<<<dim3(1), dim3(1024), 0, s>>>(cu, B, nqb, int(n_bound), blist);
      ESTP_CHECK_LAUNCH("block_list_kernel");
      const int st2 = debug_check_list(fn, blist, block_list_on_host(cu_h, B, nqb, n_bound), s);
      if (st2 != ESTP_OK) return st2;
    }
  } else if (use_list) {
    block_list_kernel<<<dim3(1), dim3(1024), 0, s>>>(cu, B, nqb, int(n_bound), blist);
  }
  const int2* bl = use_list ? blist : nullptr;
  const size_t n_rows = use_list ? n_bound : size_t(nqb) * B;  // block rows of either grid
  float lse_mul = 1.f;  // row log-sum-exps in base 2 (pass 1) ...
  if (lse_in) {         // ... or the caller's natural-log ones, converted on load
    lse2 = const_cast<float*>(lse_in);
    lse_mul = kLog2e;
  }
  if (f32) {
    launch_importance_f32(DH, static_cast<const float*>(Qv), static_cast<const float*>(Kv), cu, B, n_tok, L, Hq, Hkv,
                          nqb, c2, bl, n_rows, int(n_bound), lse_in == nullptr, lse2, lse_mul, strict, part, s);
  } else {
    const uint16_t* Q = static_cast<const uint16_t*>(Qv);
    const uint16_t* K = static_cast<const uint16_t*>(Kv);
    // GQA groups on one XCD when the grid splits into whole groups per XCD
    const size_t n_wg = n_rows * L * Hq;
    const int G = Hq / Hkv;
    const int xcd_groups = (G > 1 && n_wg % (size_t(8) * G) == 0) ? 1 : 0;
    if (!lse_in)
      attn_lse_kernel<DH><<<dim3(n_wg), dim3(kThreads), 0, s>>>(Q, K, cu, B, n_tok, L, Hq, Hkv, nqb, c2, bl,
                                                                 xcd_groups, lse2);
    attn_colsum_kernel<DH><<<dim3(n_rows * L * Hkv * nsplit), dim3(kThreads), 0, s>>>(
        Q, K, cu, B, n_tok, L, Hq, Hkv, c2, lse2, lse_mul, strict, bl, int(n_bound), nsplit, part);
  }
  LayerWeights lw{};
  if (layer_weights)
    for (int l = 0; l < L; ++l) lw.w[l] = layer_weights[l];
  attn_reduce_kernel<<<dim3((max_seqlen + 255) / 256, B), dim3(256), 0, s>>>(part, cu, n_tok, L, Hkv * nsplit, Hq,
                                                                             layer_weights ? 1 : 0, lw, S);
  ESTP_CHECK_LAUNCH(fn);
  return ESTP_OK;
}

}  // namespace detail
}  // namespace estp

using namespace estp;
using namespace estp::detail;

namespace {

// Shared argument checks of the two importance entry points.
int check_importance_args(const char* fn, const void* Q, const void* K, const int32_t* cu_seqlens, int32_t B,
                          int32_t max_seqlen, int64_t n_tok, int32_t L, int32_t Hq, int32_t Hkv, int32_t dh,
                          float scale, int dtype, float* S) {
  ESTP_REQUIRE(Q && K && cu_seqlens && S, ESTP_ERR_INVALID_ARG, "%s: Q, K, cu_seqlens and S must be non-null", fn);
  ESTP_REQUIRE(B >= 1 && max_seqlen >= 1 && L >= 1 && Hq >= 1 && Hkv >= 1, ESTP_ERR_INVALID_ARG,
               "%s: B, max_seqlen, L, Hq, Hkv must be >= 1", fn);
  ESTP_REQUIRE(n_tok >= 1 && n_tok <= INT32_MAX, ESTP_ERR_INVALID_ARG, "%s: n_tok must be in [1, 2^31), got %lld", fn,
               (long long)n_tok);
  ESTP_REQUIRE(max_seqlen <= n_tok, ESTP_ERR_INVALID_ARG, "%s: max_seqlen exceeds n_tok", fn);
  ESTP_REQUIRE(Hq % Hkv == 0, ESTP_ERR_INVALID_ARG, "%s: Hq (%d) must be a multiple of Hkv (%d)", fn, Hq, Hkv);
  ESTP_REQUIRE(scale > 0.f && scale < INFINITY, ESTP_ERR_INVALID_ARG, "%s: scale must be finite and > 0", fn);
  ESTP_REQUIRE(dtype == ESTP_BF16 || dtype == ESTP_F32, ESTP_ERR_INVALID_ARG, "%s: unknown dtype %d", fn, dtype);
  ESTP_REQUIRE(dh == 32 || dh == 64 || dh == 128, ESTP_ERR_UNSUPPORTED, "%s: head_dim %d unsupported (32, 64, 128)",
               fn, dh);
  ESTP_REQUIRE(aligned(Q, 16) && aligned(K, 16), ESTP_ERR_INVALID_ARG, "%s: Q and K must be 16-byte aligned", fn);
  ESTP_REQUIRE(size_t(L) * Hq * n_tok < (size_t(1) << 40), ESTP_ERR_INVALID_ARG, "%s: too large", fn);
  // the largest pass grid: pass 1 of the fp32 kernels, two workgroups per (block, layer, head)
  ESTP_REQUIRE(fits_launch(2 * block_rows(n_tok, B, max_seqlen) * L * Hq, kThreads) &&
                   fits_launch(size_t(B), 1) && fits_launch((size_t(max_seqlen) + 255) / 256, 256),
               ESTP_ERR_UNSUPPORTED, "%s: batch too large for one launch", fn);
  return ESTP_OK;
}

int launch_dh(const char* fn, int dh, const void* q, const void* k, bool f32, const int* cu, int B, int max_seqlen,
              int n, int L, int Hq, int Hkv, float scale, const float* lse_in, int strict, const float* lw, float* S,
              float* lse2, float* part, int2* blist, hipStream_t s) {
  switch (dh) {
    case 32:
      return launch<32>(fn, q, k, f32, cu, B, max_seqlen, n, L, Hq, Hkv, scale, lse_in, strict, lw, S, lse2, part,
                        blist, s);
    case 64:
      return launch<64>(fn, q, k, f32, cu, B, max_seqlen, n, L, Hq, Hkv, scale, lse_in, strict, lw, S, lse2, part,
                        blist, s);
    default:
      return launch<128>(fn, q, k, f32, cu, B, max_seqlen, n, L, Hq, Hkv, scale, lse_in, strict, lw, S, lse2, part,
                         blist, s);
  }
}

}  // namespace

extern "C" size_t estp_attn_importance_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t L,
                                                      int32_t Hq, int32_t Hkv, int32_t dh, int dtype) {
  (void)dh;
  if (n_tok < 1 || B < 1 || max_seqlen < 1 || L < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return 0;
  Carver c(nullptr);
  c.take<float>(size_t(L) * Hq * n_tok);   // lse2 [L, Hq, n_tok]
  c.take<float>(size_t(L) * Hkv * colsum_split(n_tok, B, max_seqlen, L, Hq, Hkv, dtype == ESTP_F32) *
                n_tok);  // column masses [L, Hkv * nsplit, n_tok]
  c.take<int2>(block_bound(n_tok, B, max_seqlen));  // list of live 256-row blocks
  return c.bytes();
}

extern "C" int estp_attn_importance(const void* Q, const void* K, const int32_t* cu_seqlens, int32_t B,
                                    int32_t max_seqlen, int64_t n_tok, int32_t L, int32_t Hq, int32_t Hkv,
                                    int32_t dh, float scale, int dtype, float* S, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  clear_error();
  const int st = check_importance_args("estp_attn_importance", Q, K, cu_seqlens, B, max_seqlen, n_tok, L, Hq, Hkv,
                                       dh, scale, dtype, S);
  if (st != ESTP_OK) return st;
  const size_t need = estp_attn_importance_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dtype);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_attn_importance: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_attn_importance: workspace must be non-null and 256-byte aligned");

  Carver c(workspace);
  float* lse2 = c.take<float>(size_t(L) * Hq * n_tok);
  float* part = c.take<float>(size_t(L) * Hkv * colsum_split(n_tok, B, max_seqlen, L, Hq, Hkv, dtype == ESTP_F32) *
                              n_tok);
  int2* blist = c.take<int2>(block_bound(n_tok, B, max_seqlen));
  return launch_dh("estp_attn_importance", dh, Q, K, dtype == ESTP_F32, cu_seqlens, B, max_seqlen, int(n_tok), L, Hq,
                   Hkv, scale, nullptr, 0, nullptr, S, lse2, part, blist, static_cast<hipStream_t>(stream));
}

extern "C" size_t estp_attn_importance_from_lse_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen,
                                                               int32_t L, int32_t Hq, int32_t Hkv, int32_t dh,
                                                               int dtype) {
  (void)dh;
  if (n_tok < 1 || B < 1 || max_seqlen < 1 || L < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return 0;
  Carver c(nullptr);
  c.take<float>(size_t(L) * Hkv * colsum_split(n_tok, B, max_seqlen, L, Hq, Hkv, dtype == ESTP_F32) *
                n_tok);  // column masses [L, Hkv * nsplit, n_tok]
  c.take<int2>(block_bound(n_tok, B, max_seqlen));  // list of live 256-row blocks
  return c.bytes();
}

extern "C" int estp_attn_importance_from_lse(const void* Q, const void* K, const float* lse,
                                             const int32_t* cu_seqlens, int32_t B, int32_t max_seqlen, int64_t n_tok,
                                             int32_t L, int32_t Hq, int32_t Hkv, int32_t dh, float scale, int dtype,
                                             float* S, void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  const int st = check_importance_args("estp_attn_importance_from_lse", Q, K, cu_seqlens, B, max_seqlen, n_tok, L,
                                       Hq, Hkv, dh, scale, dtype, S);
  if (st != ESTP_OK) return st;
  ESTP_REQUIRE(lse != nullptr, ESTP_ERR_INVALID_ARG, "estp_attn_importance_from_lse: lse must be non-null");
  const size_t need = estp_attn_importance_from_lse_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dtype);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_attn_importance_from_lse: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_attn_importance_from_lse: workspace must be non-null and 256-byte aligned");

  Carver c(workspace);
  float* part = c.take<float>(size_t(L) * Hkv * colsum_split(n_tok, B, max_seqlen, L, Hq, Hkv, dtype == ESTP_F32) *
                              n_tok);
  int2* blist = c.take<int2>(block_bound(n_tok, B, max_seqlen));
  return launch_dh("estp_attn_importance_from_lse", dh, Q, K, dtype == ESTP_F32, cu_seqlens, B, max_seqlen,
                   int(n_tok), L, Hq, Hkv, scale, lse, 0, nullptr, S, nullptr, part, blist,
                   static_cast<hipStream_t>(stream));
}

extern "C" size_t estp_attn_importance_ex_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t L,
                                                         int32_t Hq, int32_t Hkv, int32_t dh, int dtype,
                                                         int with_lse) {
  return with_lse ? estp_attn_importance_from_lse_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dtype)
                  : estp_attn_importance_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dtype);
}

extern "C" int estp_attn_importance_ex(const void* Q, const void* K, const float* lse, const int32_t* cu_seqlens,
                                       int32_t B, int32_t max_seqlen, int64_t n_tok, int32_t L, int32_t Hq,
                                       int32_t Hkv, int32_t dh, float scale, const float* layer_weights, int flags,
                                       int dtype, float* S, void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  const int st = check_importance_args("estp_attn_importance_ex", Q, K, cu_seqlens, B, max_seqlen, n_tok, L, Hq, Hkv,
                                       dh, scale, dtype, S);
  if (st != ESTP_OK) return st;
  ESTP_REQUIRE((flags & ~ESTP_IMPORTANCE_EXCLUDE_SELF) == 0, ESTP_ERR_INVALID_ARG,
               "estp_attn_importance_ex: unknown flags 0x%x", flags);
  ESTP_REQUIRE(!layer_weights || L <= kMaxWeightedLayers, ESTP_ERR_UNSUPPORTED,
               "estp_attn_importance_ex: at most %d weighted layers, got %d", kMaxWeightedLayers, L);
  if (layer_weights)
    for (int l = 0; l < L; ++l)
      ESTP_REQUIRE(layer_weights[l] == layer_weights[l] && fabsf(layer_weights[l]) < INFINITY, ESTP_ERR_INVALID_ARG,
                   "estp_attn_importance_ex: layer weight %d is not finite", l);
  const size_t need =
      estp_attn_importance_ex_workspace_size(n_tok, B, max_seqlen, L, Hq, Hkv, dh, dtype, lse != nullptr);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_attn_importance_ex: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_attn_importance_ex: workspace must be non-null and 256-byte aligned");
  Carver c(workspace);
  float* lse2 = lse ? nullptr : c.take<float>(size_t(L) * Hq * n_tok);
  float* part = c.take<float>(size_t(L) * Hkv * colsum_split(n_tok, B, max_seqlen, L, Hq, Hkv, dtype == ESTP_F32) *
                              n_tok);
  int2* blist = c.take<int2>(block_bound(n_tok, B, max_seqlen));
  return launch_dh("estp_attn_importance_ex", dh, Q, K, dtype == ESTP_F32, cu_seqlens, B, max_seqlen, int(n_tok), L,
                   Hq, Hkv, scale, lse, (flags & ESTP_IMPORTANCE_EXCLUDE_SELF) ? 1 : 0, layer_weights, S, lse2, part,
                   blist, static_cast<hipStream_t>(stream));
}
