// Token entropy, Eq. 2 (Section 4.2): H_i = -sum_v P_i(v) ln P_i(v) with
// P_i = softmax(W x_i), fused into a bf16 matrix-core GEMM so the n_tok x V
// logits never leave registers.
//
// Layout.  The GEMM is computed transposed, Z^T = W X^T: vocabulary rows are
// the MFMA "M" side (A operand, rows of W) and tokens the "N" side (B operand,
// rows of X).  Both operands are contiguous along the hidden dimension d, so
// every 16-byte transfer and every LDS fragment read is a contiguous run of 8
// bf16.  The matrix-core step is v_mfma_f32_16x16x32_bf16; in its 16 x 16
// output a lane owns one token column and 4 consecutive vocabulary rows, so
// the per-token reduction over the vocabulary runs in registers and needs
// cross-lane traffic only once, at the very end.
//
// Waves.  A workgroup is 4 waves, one per SIMD, on a 256 x 256 tile; wave
// (wv, wt) owns 128 vocabulary rows x 128 tokens as 8 x 8 blocks of 16 x 16,
// its 256 fp32 accumulators in AGPRs.  With one wave per SIMD the instruction
// stream alone decides how busy the matrix core is: every k step issues its
// 64 MFMAs with the next k step's 16 fragment reads, and after a barrier the
// 16 transfers into the freed ring slots, spaced one per four MFMAs.  The
// 16 x 16 step moves a quarter of the accumulator data per MFMA that the 32 x
// 32 step does, and under this power-limited load the chip holds a higher
// clock with it.
//
// Work split.  A workgroup owns a 256-token tile and a strided subset of the
// 256-row vocabulary tiles (vocab slice vs takes tiles vs, vs + n_vsplit, ...).
// Its steps (vocabulary tile, hidden-depth stage) form one flat sequence that
// a ring of LDS part slots prefetches straight from global memory (buffer
// loads into LDS, no register staging), across tile boundaries, so the
// folding of a finished tile into the running per-token state (max, sum
// 2^(z2-m), sum 2^(z2-m)(z2-m), base-2 units) overlaps the loads of the next
// tile.  The n_vsplit partial states per token are merged by a second small
// kernel that writes H.  When the caller asks for the most probable next
// token as well, a template variant of the kernel also keeps, per token
// column, the largest logit and its lowest vocabulary index; the same merges
// carry it (the variant without it is the plain kernel).
//
// XCDs.  Workgroup ids are remapped so the 32 workgroups resident on one XCD
// (ids are dealt round-robin over the 8 XCDs) cover 4 vocabulary slices x 8
// token tiles, and one dispatch wave of 256 covers 16 x 16: concurrent
// workgroups stream the same W and X tiles through that XCD's L2.  An XCD
// takes the slices g, g+4, g+8, g+12, so the slices that hold one tile more
// than the others are spread over the XCDs.
#include <atomic>
#include <mutex>

#include "estp_common.h"
#include "f32_paths.h"

namespace estp {
namespace detail {

constexpr int kBV = 256;       // vocabulary rows per tile
constexpr int kBT = 256;       // tokens per tile
constexpr int kWaves = 4;      // waves per workgroup, one per SIMD
constexpr int kMaxVsplit = 16;
constexpr int kNB = 8;         // 16-row blocks per wave, both operands (128 rows each)
constexpr int kMfmaPerStep = kNB * kNB;

// Geometry of one LDS stage (kBV rows of W, kBT rows of X, BK bf16 of the
// hidden dimension each).  BK = 64 makes every row of a stage one 128-byte run
// of global memory, which the texture path fetches as a single request; BK =
// 32 (64-byte runs) serves hidden sizes that are an odd multiple of 32.
template <int BK>
struct Geom {
  static constexpr int kSub = BK / 32;                              // 32-deep MFMA steps per stage
  static constexpr int kRowBytes = BK * 2;                          // 64 or 128 B
  static constexpr int kChunks = kRowBytes / 16;                    // 16-byte chunks per row
  static constexpr int kRowsPerInst = 64 / kChunks;                 // rows per wave transfer (1 KB)
  static constexpr int L = kBV / (kRowsPerInst * kWaves);           // transfers per wave per part
  static constexpr int kPartBytes = kBV * kRowBytes;                // one operand of one stage (kBV == kBT)
  static constexpr int kRowsPerWindow = 256 / kRowBytes;            // rows that share a 256-byte bank window
  // Chunk swizzle: the 16 rows that 16 consecutive lanes read at one logical
  // chunk land in 16 distinct 16-byte bank groups.  It depends on the row only
  // through (row / kRowsPerWindow) % kChunks, which repeats every 16 rows.
  __device__ static __forceinline__ int swz(int row, int chunk) {
    return chunk ^ ((row / kRowsPerWindow) & (kChunks - 1));
  }
};

// Spacing of the instructions threaded between the 64 MFMAs of a k step:
// fragment read q after MFMA kReadEvery * q, transfer t after MFMA
// kDmaFirst + kDmaEvery * t.  Evenly spread, neither kind ever holds the wave
// away from the matrix core for long (measured: reading all 16 fragments over
// the first 16 MFMAs ran ~6% slower).
constexpr int kReadEvery = 4, kDmaFirst = 2, kDmaEvery = 4;
constexpr int kSetupA = 5, kSetupB = 37;  // MFMAs after which the next parts' scalar set-up runs

__device__ __forceinline__ f32x4_t mfma16(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Largest logit with its vocabulary index: b wins over a when it is larger, or
// equal with a lower index (ties go to the lowest index).
__device__ __forceinline__ void arg_merge(float& av, int& ai, float bv, int bi) {
  const bool take = (bv > av) | ((bv == av) & (bi < ai));  // no short circuit: no branches
  av = take ? bv : av;
  ai = take ? bi : ai;
}

// A stage is BK deep (kSub k steps).  Ring of P part slots: part 2s + 0 / 2s + 1
// (W / X of stage s) lives in slot (2s + o) % P.  Within a stage the wave runs
// kSub k steps, each reading the next step's fragments while its MFMAs run.
// Before the last k step every wave waits for its own fragment reads (so stage
// s is no longer read) and for stage s + 1 to have landed, then one barrier;
// after it the two freed slots take parts 2s + P and 2s + P + 1.  With P odd
// the W part of a stage is issued one stage before its X part, and about
// (P - 2) / 2 stages of loads are in flight while a stage is consumed.
template <int P, int BK, bool kArg>
__global__ __launch_bounds__(kWaves * 64, 1) void entropy_gemm_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, int n_tok, int d, int V, int n_vsplit,
    int n_vt, int n_tt, float* __restrict__ part_m, float* __restrict__ part_s, float* __restrict__ part_t,
    float* __restrict__ part_zmax, int* __restrict__ part_arg) {
  using G = Geom<BK>;
  constexpr int L = G::L;
  constexpr int kSub = G::kSub;
  constexpr int kBlockBytes = 16 * G::kRowBytes;
  static_assert(P >= 4 && P % 2 == 1, "the ring needs two stages and an odd slot count");
  static_assert(kReadEvery * (2 * kNB - 1) < kMfmaPerStep, "fragment reads fit in a k step");
  static_assert(kDmaFirst + kDmaEvery * (2 * L - 1) < kMfmaPerStep, "transfers fit in a k step");
  __shared__ __attribute__((aligned(16))) char lds[P * G::kPartBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave & 1;   // which 128-row half of the vocabulary tile
  const int wt = wave >> 1;  // which 128-token half of the token tile

  // ---- workgroup -> (vocabulary slice, token tile)
  int vs, tt;
  {
    const int bid = blockIdx.x;
    constexpr int R = 32;  // workgroups resident on one XCD
    // whole dispatch waves of 16 token tiles x 16 slices take the XCD-aware order; the
    // token tiles past the last whole group of 16 (ragged batches) follow in plain order
    const int n_full = n_vsplit == 16 ? (n_tt / (R / 2)) * (R / 2) * 16 : 0;
    if (bid < n_full) {
      const int xcd = bid & 7, j = bid >> 3;
      const int wave_idx = j / R, jj = j % R;
      vs = (jj & 3) * 4 + (xcd & 3);
      tt = wave_idx * (R / 2) + (xcd >> 2) * (R / 4) + (jj >> 2);
    } else {
      const int r = bid - n_full;
      vs = r % n_vsplit;
      tt = n_full / n_vsplit + r / n_vsplit;
    }
  }
  const int nk = d / BK;
  const int n_my_tiles = (n_vt - vs + n_vsplit - 1) / n_vsplit;
  const size_t row_stride = size_t(d) * 2;  // bytes per row of W and X

  // ---- staging: lane l of transfer i fills row kRowsPerInst*(kWaves i + wave) + l / kChunks,
  // physical chunk l % kChunks, i.e. logical chunk swz(row, l % kChunks) of that row.  The
  // transfers go through buffer resources that cover exactly the live rows of a tile (W: the
  // vocabulary tile, X: the token tile), so rows past V or n_tok read as zero with no clamping;
  // each transfer is one instruction: per-lane byte offset in the tile (fixed for the whole
  // kernel) + the stage's depth offset in a scalar register.
  uint32_t st_off[L];
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const int row = G::kRowsPerInst * (kWaves * i + wave) + lane / G::kChunks;
    st_off[i] = uint32_t(row) * uint32_t(row_stride) + uint32_t(G::swz(row, lane % G::kChunks) * 16);
  }
  const uint32_t tile_bytes = uint32_t(kBV) * uint32_t(row_stride);
  const buf_rsrc_t rx = make_rsrc(reinterpret_cast<const char*>(X) + size_t(tt) * kBT * row_stride,
                                  uint32_t(min(kBT, n_tok - tt * kBT)) * uint32_t(row_stride));

  // ---- prefetch of parts in order 0, 1, 2, ...: part q is operand q % 2 of
  // stage q / 2 = (tile, ks).  Parts past the end are issued with an empty
  // resource (no memory access, zeros into the slot being freed, never read),
  // so every barrier issues exactly 2 L transfers per wave and the waits below
  // are the same on every stage; the loop body stays one basic block.
  int pf_tile = 0, pf_ks = 0, pf_slot = 0, pf_op = 0;
  int pf_vt = vs;                                                                  // vocabulary tile of the prefetch
  const char* pf_w = reinterpret_cast<const char*>(W) + size_t(vs) * tile_bytes;  // its rows of W
  const size_t w_step = size_t(n_vsplit) * tile_bytes;
  const buf_rsrc_t r_none = make_rsrc(X, 0u);
  struct Part {
    buf_rsrc_t rsrc;  // the vocabulary tile's rows of W, or the token tile's rows of X
    uint32_t soff;    // depth offset of the stage inside a row
    char* dst;        // this wave's first 1 KB block of the slot
  };
  // Source and destination of the next part; advances the part counters.
  auto next_part = [&](int op) {
    const bool live = pf_tile < n_my_tiles;
    Part p;
    p.dst = lds + pf_slot * G::kPartBytes + G::kRowsPerInst * wave * G::kRowBytes;
    p.soff = uint32_t(pf_ks) * G::kRowBytes;
    if (op == 0) {
      // past the last tile pf_w points beyond W, but the empty resource never reads it
      const uint32_t rows = live ? uint32_t(min(kBV, V - pf_vt * kBV)) : 0u;
      p.rsrc = make_rsrc(pf_w, rows * uint32_t(row_stride));
    } else {
      p.rsrc = live ? rx : r_none;
      const bool wrap = pf_ks + 1 == nk;
      pf_ks = wrap ? 0 : pf_ks + 1;
      if (wrap) {
        ++pf_tile;
        pf_vt += n_vsplit;
        pf_w += w_step;
      }
    }
    pf_slot = pf_slot + 1 == P ? 0 : pf_slot + 1;
    return p;
  };
  // Transfer i (of L) of a part: 1 KB, kRowsPerInst rows.
  auto dma_one = [&](const Part& p, int i) {
    lds_dma16_buf(p.rsrc, st_off[i], p.soff, p.dst + G::kRowsPerInst * kWaves * i * G::kRowBytes);
  };
  auto issue_part = [&]() {
    const Part p = next_part(pf_op);
#pragma unroll
    for (int i = 0; i < L; ++i) dma_one(p, i);
    pf_op ^= 1;
  };
  // The two parts issued at every barrier: their operands are fixed, since an
  // even number of parts precedes each barrier's pair.
  constexpr int kOpA = P % 2, kOpB = kOpA ^ 1;

  // ---- fragment reads: lane (r = lane % 16, q = lane / 16) reads 8 bf16 at k offset
  // 32 kk + 8 q of row r of each 16-row block.  The swizzle is the same in every
  // 16-row block, so one offset per k step serves all 8 blocks, 16 rows apart.
  const int fr = lane & 15, fq = lane >> 4;
  uint32_t fa_off[kSub], fb_off[kSub];
#pragma unroll
  for (int kk = 0; kk < kSub; ++kk) {
    const int ra = wv * 128 + fr, rb = wt * 128 + fr;
    fa_off[kk] = ra * G::kRowBytes + G::swz(ra, kk * 4 + fq) * 16;
    fb_off[kk] = rb * G::kRowBytes + G::swz(rb, kk * 4 + fq) * 16;
  }
  struct Frags {
    bf16x8_t a[kNB], b[kNB];  // vocabulary-row blocks, token blocks
  };
  // fragment q of 2 kNB: the A blocks first, then the B blocks
  auto read_frag = [&](Frags& f, int slot_w, int slot_x, int kk, int q) {
    if (q < kNB)
      f.a[q] = *reinterpret_cast<const bf16x8_t*>(lds + slot_w * G::kPartBytes + fa_off[kk] + q * kBlockBytes);
    else
      f.b[q - kNB] = *reinterpret_cast<const bf16x8_t*>(lds + slot_x * G::kPartBytes + fb_off[kk] +
                                                        (q - kNB) * kBlockBytes);
  };

  // ---- per-lane entropy state for the kNB token columns this lane owns
  Ent2 st[kNB];
#pragma unroll
  for (int j = 0; j < kNB; ++j) st[j] = Ent2{-INFINITY, 0.f, 0.f};
  // mode tracking (kArg): the largest logit seen per token column and its vocabulary index.
  // The four lanes fq = 0..3 that share a column merge their candidates after every tile,
  // and lane fq keeps columns 2 fq and 2 fq + 1 only: 4 registers instead of 16, which the
  // fold's register budget needs.
  float zmax[2] = {-INFINITY, -INFINITY};
  int zarg[2] = {INT32_MAX, INT32_MAX};

  // ---- prologue: the first parts in flight; wait for stage 0, read its first fragments
#pragma unroll
  for (int q = 0; q < P; ++q) issue_part();
  wait_vm<(P - 2) * L>();
  lds_barrier();
  // With two k steps per stage the buffers alternate inside the stage and stage
  // s + 1 starts in f[0]; with one, each stage starts by moving the fragments
  // read during the previous stage from f[1] into f[0].
  Frags f[2];
  constexpr int kFirst = kSub == 1 ? 1 : 0;
#pragma unroll
  for (int q = 0; q < 2 * kNB; ++q) read_frag(f[kFirst], 0, 1, 0, q);
  int sw = 0;  // slot of the W part of the current stage; its X part is in sw + 1 (mod P)

  for (int tile = 0; tile < n_my_tiles; ++tile) {
    f32x4_t acc[kNB][kNB];
#pragma unroll
    for (int i = 0; i < kNB; ++i)
#pragma unroll
      for (int j = 0; j < kNB; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int ks = 0; ks < nk; ++ks) {
      const int sx = sw + 1 == P ? 0 : sw + 1;
      const int sw_next = sx + 1 == P ? 0 : sx + 1;
      const int sx_next = sw_next + 1 == P ? 0 : sw_next + 1;
      Part pa, pb;  // the two parts issued after this stage's barrier
#pragma unroll
      for (int u = 0; u < kSub; ++u) {
        Frags& cur = f[u & 1];
        Frags& nxt = f[(u + 1) & 1];
        const bool last = u + 1 == kSub;
        if (last) {
          // This wave's reads of the stage are done (lgkmcnt 0 inside the
          // barrier) and the next stage has landed (only the P - 4 parts
          // issued after it may still be in flight): after the barrier nobody
          // reads this stage's slots again, so they take the next two parts.
          if (kSub == 1) {
            pa = next_part(kOpA);
            pb = next_part(kOpB);
          }
          __builtin_amdgcn_sched_barrier(0);
          wait_vm<(P - 4) * L>();
          lds_barrier();
          if (kSub == 1) f[0] = f[1];
        }
        // the MFMAs of this k step, with the next k step's fragment reads (past
        // the last stage: read and never used) and, after the barrier, the
        // transfers into the freed slots threaded between them
#pragma unroll
        for (int i = 0; i < kNB; ++i)
#pragma unroll
          for (int j = 0; j < kNB; ++j) {
            const int m = i * kNB + j;
            acc[i][j] = mfma16(cur.a[i], cur.b[j], acc[i][j]);
            // scalar set-up of the parts issued after the coming barrier, each behind
            // an MFMA of the k step before it
            if (u + 2 == kSub && m == kSetupA) pa = next_part(kOpA);
            if (u + 2 == kSub && m == kSetupB) pb = next_part(kOpB);
            if (m % kReadEvery == 0 && m / kReadEvery < 2 * kNB) {
              if (last)
                read_frag(nxt, sw_next, sx_next, 0, m / kReadEvery);
              else
                read_frag(nxt, sw, sx, u + 1, m / kReadEvery);
            }
            if (last && m >= kDmaFirst && (m - kDmaFirst) % kDmaEvery == 0 && (m - kDmaFirst) / kDmaEvery < 2 * L) {
              const int t = (m - kDmaFirst) / kDmaEvery;
              if (t < L)
                dma_one(pa, t);
              else
                dma_one(pb, t - L);
            }
            __builtin_amdgcn_sched_barrier(0);
          }
      }
      sw = sw_next;
    }

    // ---- fold the finished tile into the running states.  acc[i][j][r] is the
    // logit of vocabulary row vt*256 + wv*128 + 16 i + 4 fq + r for token
    // tt*256 + wt*128 + 16 j + fr.
    //
    // The state (m, s, t) is kept relative to a reference m that is the running
    // log-sum-exp after each tile (rebased so that s = 1).  Full tiles are then
    // folded with 3 VALU ops and one exp2 per logit and no max pass; a tile whose
    // logits exceed the reference by more than 2^64 in weight (or overflow) is
    // refolded exactly with its own max.  The ragged last vocabulary tile always
    // takes the exact, masked path.
    const int vt = vs + tile * n_vsplit;
    const bool ragged = (vt + 1) * kBV > V;
    const int lim = V - (vt * kBV + wv * 128 + 4 * fq);  // live rows: 16 i + r < lim
#pragma unroll
    for (int j = 0; j < kNB; ++j) {
      Ent2 e = st[j];
      bool exact = ragged;
      if (!ragged) {
        if (tile == 0) {  // first tile: the tile's own max is the reference
          float mx = acc[0][j][0];
#pragma unroll
          for (int i = 0; i < kNB; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) mx = fmaxf(mx, acc[i][j][r]);
          e = Ent2{mx * kLog2e, 0.f, 0.f};
        }
        float s = e.s, t = e.t;
#pragma unroll
        for (int i = 0; i < kNB; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float dd = fmaf(acc[i][j][r], kLog2e, -e.m);
            const float p = fast_exp2(dd);
            s += p;
            t = fmaf(p, dd, t);
          }
        if (s <= 0x1p64f) {
          e.s = s;
          e.t = t;
        } else {
          exact = true;  // overflow (or a logit far above the reference): refold exactly
        }
      }
      if (exact) {
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < kNB; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const bool live = !ragged || i * 16 + r < lim;
            mx = live ? fmaxf(mx, acc[i][j][r]) : mx;
          }
        const float mnew = fmaxf(e.m, mx * kLog2e);
        const float dl = fmaxf(e.m - mnew, kExp2Floor);
        const float sc = fast_exp2(dl);
        float s = sc * e.s;
        float t = sc * (e.t + e.s * dl);
#pragma unroll
        for (int i = 0; i < kNB; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            // dead rows enter as -inf: dd clamps to the floor and adds 0 * floor,
            // also while mnew is still -inf (a lane with no live row yet)
            const bool live = !ragged || i * 16 + r < lim;
            const float dd = fmaxf(fmaf(live ? acc[i][j][r] : -INFINITY, kLog2e, -mnew), kExp2Floor);
            const float p = fast_exp2(dd);
            s += p;
            t = fmaf(p, dd, t);
          }
        e = Ent2{mnew, s, t};
      }
      // rebase to the running log-sum-exp: m += log2 s, s = 1, t = t / s - log2 s
      // (s >= 1 here: the reference never exceeds the largest logit seen, in base 2)
      if (e.s > 0.f) {
        const float dl = fast_log2(e.s);
        e = Ent2{e.m + dl, 1.f, e.t / e.s - dl};
      }
      st[j] = e;
    }
    if (kArg) {
      // the next-token mode, in a loop of its own so that the eight columns' independent compare
      // chains interleave.  Per column: the tile's largest live logit, then the lowest of the
      // lane's rows holding it (rows visited from the last to the first, the last match kept;
      // ordinals 4 i + r are small constants, no literal moves).  Dead rows of the ragged tile
      // lie after every live row, so an equal dead row never wins.  No branches inside: every
      // compare feeds its select.
      float tb[kNB];
#pragma unroll
      for (int j = 0; j < kNB; ++j) tb[j] = -INFINITY;
      if (ragged) {
#pragma unroll
        for (int j = 0; j < kNB; ++j)
#pragma unroll
          for (int i = 0; i < kNB; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) tb[j] = fmaxf(tb[j], i * 16 + r < lim ? acc[i][j][r] : -INFINITY);
      } else {
#pragma unroll
        for (int j = 0; j < kNB; ++j)
#pragma unroll
          for (int i = 0; i < kNB; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) tb[j] = fmaxf(tb[j], acc[i][j][r]);
      }
#pragma unroll
      for (int j = 0; j < kNB; ++j) {
        int k = 0;
#pragma unroll
        for (int i = kNB - 1; i >= 0; --i)
#pragma unroll
          for (int r = 3; r >= 0; --r) k = acc[i][j][r] == tb[j] ? 4 * i + r : k;
        // the column's candidate over the four lanes that share it, then kept by lane j / 2
        float cb = tb[j];
        int ci = vt * kBV + wv * 128 + 4 * fq + (k >> 2) * 16 + (k & 3);
#pragma unroll
        for (int o = 16; o <= 32; o <<= 1) arg_merge(cb, ci, __shfl_xor(cb, o, 64), __shfl_xor(ci, o, 64));
        const bool keep = (fq == j / 2) & (cb > zmax[j & 1]);  // strict: an earlier tile keeps equal maxima
        zmax[j & 1] = keep ? cb : zmax[j & 1];
        zarg[j & 1] = keep ? ci : zarg[j & 1];
      }
    }
  }  // tile

  // ---- lanes l, l ^ 16, l ^ 32 and l ^ 48 hold the same tokens: merge them
#pragma unroll
  for (int j = 0; j < kNB; ++j) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      Ent2 x;
      x.m = __shfl_xor(st[j].m, o, 64);
      x.s = __shfl_xor(st[j].s, o, 64);
      x.t = __shfl_xor(st[j].t, o, 64);
      st[j] = ent2_merge(st[j], x);
    }
  }
  // ---- the two vocabulary halves (wv = 0, 1) hold the same tokens: merge through LDS.
  // The transfers issued at the last barrier (empty parts past the end, which still write
  // zeros into their slots) must land before slot 0 is reused.
  wait_vm<0>();
  __syncthreads();  // every wave is done with the ring and no transfer remains in flight
  constexpr int kSt = kArg ? 5 : 3;                // floats per token in the exchange
  float* xbuf = reinterpret_cast<float*>(lds);  // [BT tokens][kSt]
  if (wv == 1 && fq == 0) {
#pragma unroll
    for (int j = 0; j < kNB; ++j) {
      float* p = xbuf + (wt * 128 + j * 16 + fr) * kSt;
      p[0] = st[j].m;
      p[1] = st[j].s;
      p[2] = st[j].t;
    }
  }
  if (kArg && wv == 1) {  // lane fq holds columns 2 fq and 2 fq + 1
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      float* p = xbuf + (wt * 128 + (2 * fq + c) * 16 + fr) * kSt;
      p[3] = zmax[c];
      p[4] = __int_as_float(zarg[c]);
    }
  }
  __syncthreads();
  if (wv == 0 && fq == 0) {
#pragma unroll
    for (int j = 0; j < kNB; ++j) {
      const int tl = wt * 128 + j * 16 + fr;
      const float* p = xbuf + tl * kSt;
      Ent2 r = ent2_merge(st[j], Ent2{p[0], p[1], p[2]});
      const int tok = tt * kBT + tl;
      if (tok < n_tok) {
        const size_t o = size_t(vs) * n_tok + tok;
        part_m[o] = r.m;
        part_s[o] = r.s;
        part_t[o] = r.t;
      }
    }
  }
  if (kArg && wv == 0) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int tl = wt * 128 + (2 * fq + c) * 16 + fr;
      const int tok = tt * kBT + tl;
      if (tok < n_tok) {
        const float* p = xbuf + tl * kSt;
        float zb = zmax[c];
        int ib = zarg[c];
        arg_merge(zb, ib, p[3], __float_as_int(p[4]));
        const size_t o = size_t(vs) * n_tok + tok;
        part_zmax[o] = zb;
        part_arg[o] = ib;
      }
    }
  }
}

// Merge the n_vsplit partial states of each token and write H in nats:
// H = ln2 * (log2 s - t / s).  With `arg` non-null, also the vocabulary index
// of the largest logit over the slices (lowest index among equal maxima).
__global__ __launch_bounds__(256) void entropy_merge_kernel(const float* __restrict__ part_m,
                                                            const float* __restrict__ part_s,
                                                            const float* __restrict__ part_t,
                                                            const float* __restrict__ part_zmax,
                                                            const int* __restrict__ part_arg, int n_tok,
                                                            int n_vsplit, float* __restrict__ H,
                                                            int32_t* __restrict__ arg) {
  const int tok = blockIdx.x * 256 + threadIdx.x;
  if (tok >= n_tok) return;
  Ent2 a{part_m[tok], part_s[tok], part_t[tok]};
  for (int v = 1; v < n_vsplit; ++v) {
    const size_t o = size_t(v) * n_tok + tok;
    a = ent2_merge(a, Ent2{part_m[o], part_s[o], part_t[o]});
  }
  H[tok] = kLn2 * (fast_log2(a.s) - a.t / a.s);
  if (arg) {
    float zb = part_zmax[tok];
    int ib = part_arg[tok];
    for (int v = 1; v < n_vsplit; ++v) {
      const size_t o = size_t(v) * n_tok + tok;
      arg_merge(zb, ib, part_zmax[o], part_arg[o]);
    }
    arg[tok] = ib;
  }
}

int choose_vsplit(int n_vt) { return n_vt < kMaxVsplit ? n_vt : kMaxVsplit; }

}  // namespace detail
}  // namespace estp

using namespace estp;
using namespace estp::detail;

extern "C" size_t estp_token_entropy_workspace_size(int64_t n_tok, int32_t d, int32_t V, int dtype) {
  (void)d;
  (void)dtype;
  if (n_tok < 1 || V < 1) return 0;
  const int n_vt = (V + kBV - 1) / kBV;
  Carver c(nullptr);
  // per-slice (m, s, t) states, then the per-slice largest logit and its index
  for (int i = 0; i < 5; ++i) c.take<float>(size_t(choose_vsplit(n_vt)) * n_tok);
  return c.bytes();
}

namespace {

// Host-side checks shared by both entry points; `fn` names the caller in the error message.
int check_entropy_args(const char* fn, const void* X, const void* W, int64_t n_tok, int32_t d, int32_t V,
                       int dtype, const float* H, const int32_t* vocab_argmax) {
  ESTP_REQUIRE(X && W && H, ESTP_ERR_INVALID_ARG, "%s: X, W and H must be non-null", fn);
  ESTP_REQUIRE(n_tok >= 1 && n_tok <= INT32_MAX, ESTP_ERR_INVALID_ARG, "%s: n_tok must be in [1, 2^31), got %lld", fn,
               (long long)n_tok);
  ESTP_REQUIRE(V >= 1, ESTP_ERR_INVALID_ARG, "%s: V must be >= 1, got %d", fn, V);
  ESTP_REQUIRE(d >= 8 && d % 8 == 0, ESTP_ERR_INVALID_ARG, "%s: d must be a positive multiple of 8, got %d", fn, d);
  ESTP_REQUIRE(dtype == ESTP_BF16 || dtype == ESTP_F32, ESTP_ERR_INVALID_ARG, "%s: unknown dtype %d", fn, dtype);
  ESTP_REQUIRE(dtype == ESTP_F32 || d % 32 == 0, ESTP_ERR_UNSUPPORTED,
               "%s: d must be a multiple of 32 for the matrix-core path, got %d", fn, d);
  ESTP_REQUIRE(size_t(d) * 2 * kBV < (size_t(1) << 32), ESTP_ERR_UNSUPPORTED, "%s: d = %d too large", fn, d);
  ESTP_REQUIRE(aligned(X, 16) && aligned(W, 16), ESTP_ERR_INVALID_ARG, "%s: X and W must be 16-byte aligned", fn);
  ESTP_REQUIRE(aligned(H, 4) && aligned(vocab_argmax, 4), ESTP_ERR_INVALID_ARG,
               "%s: H and vocab_argmax must be 4-byte aligned", fn);
  const int n = int(n_tok);
  const int n_vsplit = choose_vsplit((V + kBV - 1) / kBV);
  const size_t n_wg =
      dtype == ESTP_F32 ? entropy_f32_workgroups(n, n_vsplit) : size_t(n_vsplit) * size_t((n + kBT - 1) / kBT);
  ESTP_REQUIRE(fits_launch(n_wg, kWaves * 64), ESTP_ERR_UNSUPPORTED,
               "%s: n_tok = %d needs %zu workgroups, more than one launch holds", fn, n, n_wg);
  return ESTP_OK;
}

// The kernels of one call on checked arguments; `workspace` holds
// estp_token_entropy_workspace_size() bytes, 256-byte aligned.
int launch_token_entropy(const void* X, const void* W, int n, int d, int V, int dtype, float* H,
                         int32_t* vocab_argmax, void* workspace, hipStream_t s) {
  const int n_vt = (V + kBV - 1) / kBV;
  const int n_tt = (n + kBT - 1) / kBT;
  const int n_vsplit = choose_vsplit(n_vt);
  Carver c(workspace);
  float* pm = c.take<float>(size_t(n_vsplit) * n);
  float* ps = c.take<float>(size_t(n_vsplit) * n);
  float* pt = c.take<float>(size_t(n_vsplit) * n);
  float* pz = c.take<float>(size_t(n_vsplit) * n);
  int* pa = c.take<int>(size_t(n_vsplit) * n);
  const bool want_arg = vocab_argmax != nullptr;

  if (dtype == ESTP_F32) {
    launch_entropy_f32(static_cast<const float*>(X), static_cast<const float*>(W), n, d, V, n_vsplit, pm, ps, pt, pz,
                       want_arg ? pa : nullptr, s);
    ESTP_CHECK_LAUNCH("entropy_f32_kernel");
  } else {
    const dim3 grid(n_vsplit * n_tt), block(kWaves * 64);
    const uint16_t* Xh = static_cast<const uint16_t*>(X);
    const uint16_t* Wh = static_cast<const uint16_t*>(W);
    if (d % 64 == 0) {
      if (want_arg)
        entropy_gemm_kernel<5, 64, true><<<grid, block, 0, s>>>(Xh, Wh, n, d, V, n_vsplit, n_vt, n_tt, pm, ps, pt, pz,
                                                                pa);
      else
        entropy_gemm_kernel<5, 64, false><<<grid, block, 0, s>>>(Xh, Wh, n, d, V, n_vsplit, n_vt, n_tt, pm, ps, pt,
                                                                 nullptr, nullptr);
    } else {
      if (want_arg)
        entropy_gemm_kernel<9, 32, true><<<grid, block, 0, s>>>(Xh, Wh, n, d, V, n_vsplit, n_vt, n_tt, pm, ps, pt, pz,
                                                                pa);
      else
        entropy_gemm_kernel<9, 32, false><<<grid, block, 0, s>>>(Xh, Wh, n, d, V, n_vsplit, n_vt, n_tt, pm, ps, pt,
                                                                 nullptr, nullptr);
    }
    ESTP_CHECK_LAUNCH("entropy_gemm_kernel");
  }
  entropy_merge_kernel<<<dim3((n + 255) / 256), dim3(256), 0, s>>>(pm, ps, pt, pz, want_arg ? pa : nullptr, n,
                                                                   n_vsplit, H, vocab_argmax);
  ESTP_CHECK_LAUNCH("entropy_merge_kernel");
  return ESTP_OK;
}

}  // namespace

extern "C" int estp_token_entropy(const void* X, const void* W, int64_t n_tok, int32_t d, int32_t V, int dtype,
                                  float* H, int32_t* vocab_argmax, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  clear_error();
  const int st = check_entropy_args("estp_token_entropy", X, W, n_tok, d, V, dtype, H, vocab_argmax);
  if (st != ESTP_OK) return st;
  const size_t need = estp_token_entropy_workspace_size(n_tok, d, V, dtype);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_token_entropy: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_token_entropy: workspace must be non-null and 256-byte aligned");
  return launch_token_entropy(X, W, int(n_tok), d, V, dtype, H, vocab_argmax, workspace,
                              static_cast<hipStream_t>(stream));
}


// ------------------------------------------------------------------ no-allocation variant
//
// The per-slice partial states of estp_token_entropy_noalloc live in this
// file-scope device array instead of a caller workspace.  Every GPU the
// library runs on holds its own copy until the process ends.  In host code
// the array's name is only a stand-in: the device address of the current
// GPU's copy comes from hipGetSymbolAddress, looked up once per device and
// kept; kernels and copies only ever see that address.  Every partial is
// written before it is read, so nothing has to be cleared between calls;
// calls that overlap on one GPU share the array and race.
static_assert(ESTP_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");
static __device__ __align__(256) char scratch[ESTP_NOALLOC_SCRATCH_BYTES];

namespace {

std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current GPU's `scratch` (nullptr and an error message on failure).
void* scratch_of_current_device(const char* fn) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_error("%s: no usable current HIP device (%d)", fn, dev);
    return nullptr;
  }
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch[dev].load(std::memory_order_relaxed);
  if (!p) {
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_error("%s: hipGetSymbolAddress of the scratch array on device %d: %s", fn, dev, hipGetErrorString(e));
      return nullptr;
    }
    g_scratch[dev].store(p, std::memory_order_release);
  }
  return p;
}

}  // namespace

extern "C" int estp_token_entropy_noalloc(const void* X, const void* W, int64_t n_tok, int32_t d, int32_t V,
                                          int dtype, float* H, int32_t* vocab_argmax, void* stream) {
  clear_error();
  const char* fn = "estp_token_entropy_noalloc";
  const int st = check_entropy_args(fn, X, W, n_tok, d, V, dtype, H, vocab_argmax);
  if (st != ESTP_OK) return st;
  const size_t need = estp_token_entropy_workspace_size(n_tok, d, V, dtype);
  ESTP_REQUIRE(need <= size_t(ESTP_NOALLOC_SCRATCH_BYTES), ESTP_ERR_UNSUPPORTED,
               "%s: n_tok = %lld with V = %d needs %zu bytes of scratch, more than the %zu the library holds per "
               "GPU; call estp_token_entropy with a workspace instead",
               fn, (long long)n_tok, V, need, size_t(ESTP_NOALLOC_SCRATCH_BYTES));
  void* ws = scratch_of_current_device(fn);
  if (!ws) return ESTP_ERR_HIP;
  return launch_token_entropy(X, W, int(n_tok), d, V, dtype, H, vocab_argmax, ws, static_cast<hipStream_t>(stream));
}
