// Token entropy, Eq. 2 (Section 4.2): H_i = -sum_v P_i(v) ln P_i(v) with
// P_i = softmax(W x_i), fused into a bf16 matrix-core GEMM so the n_tok x V
// logits never leave registers.
//
// Layout.  The GEMM is computed transposed, Z^T = W X^T: vocabulary rows are
// the MFMA "M" side (A operand, rows of W) and tokens the "N" side (B operand,
// rows of X).  Both operands are contiguous along the hidden dimension d, so
// every 16-byte global load and every LDS fragment read is a contiguous run
// of 8 bf16.  In the 32x32 MFMA output a lane owns one token column and 16
// vocabulary rows, so the per-token reduction over the vocabulary runs in
// registers with no cross-lane traffic until the very end.
//
// Work split.  A workgroup owns a 256-token tile and a strided subset of the
// 256-row vocabulary tiles (vocab slice vs takes tiles vs, vs + n_vsplit, ...).
// Its steps (vocabulary tile, hidden-depth stage) form one flat sequence that
// an S-deep LDS ring prefetches straight from global memory
// (global_load_lds_dwordx4, no register staging), across tile boundaries, so
// the folding of a finished 256 x 256 tile into the running per-token state
// (max, sum 2^(z2-m), sum 2^(z2-m)(z2-m), base-2 units) overlaps the loads of
// the next tile.  The n_vsplit partial states per token are merged by a
// second small kernel that writes H.  Workgroup ids are remapped so the 32
// workgroups resident on one XCD (ids are dealt round-robin over the 8 XCDs)
// cover 4 vocabulary slices x 8 token tiles, and one dispatch wave of 256
// covers 16 x 16: concurrent workgroups stream the same W and X tiles through
// that XCD's L2.  An XCD takes the slices g, g+4, g+8, g+12, so the slices
// that hold one tile more than the others are spread over the XCDs.
#include "estp_common.h"

namespace estp {
namespace detail {

constexpr int kBV = 256;       // vocabulary rows per tile
constexpr int kBT = 256;       // tokens per tile
constexpr int kWaves = 8;      // waves per workgroup, two per SIMD
constexpr int kMaxVsplit = 16;

// Geometry of one LDS stage (kBV rows of W then kBT rows of X, BK bf16 of the
// hidden dimension each) and of the wave layout: waves split the 256 x 256
// tile 2 (vocabulary) x 4 (tokens); a wave owns 128 vocabulary rows x 64 tokens.
// BK = 64 makes every row of a stage one 128-byte run of global memory, which
// the texture path fetches as a single request; BK = 32 (64-byte runs) serves
// hidden sizes that are an odd multiple of 32.
template <int BK>
struct Geom {
  static constexpr int kThreads = kWaves * 64;
  static constexpr int TW = 2 * kBT / kWaves;                       // 64 tokens per wave
  static constexpr int JT = TW / 32;                                // 32-token MFMA blocks per wave
  static constexpr int kSub = BK / 16;                              // 16-deep MFMA steps per stage
  static constexpr int kRowBytes = BK * 2;                          // 64 or 128 B
  static constexpr int kChunks = kRowBytes / 16;                    // 16-byte chunks per row
  static constexpr int kRowsPerInst = 64 / kChunks;                 // rows per wave instruction (1 KB)
  static constexpr int kInstW = kBV / (kRowsPerInst * kWaves);      // W transfers per wave per stage
  static constexpr int kInstX = kBT / (kRowsPerInst * kWaves);      // X transfers per wave per stage
  static constexpr int kLoadsPerStage = kInstW + kInstX;            // vector-memory instructions per wave
  static constexpr int kPartBytes = kBV * kRowBytes;                // one operand of one stage (kBV == kBT)
  static constexpr int kRowsPerWindow = 256 / kRowBytes;            // rows that share a 256-byte bank window
  // Chunk swizzle: the 16 rows that 16 consecutive lanes read at one logical
  // chunk land in 16 distinct 16-byte bank groups.
  __device__ static __forceinline__ int swz(int row, int chunk) {
    return chunk ^ ((row / kRowsPerWindow) & (kChunks - 1));
  }
};

// One 16-deep k step of a wave's tile: 4 A fragments (vocabulary rows) and
// JT B fragments (tokens), 8 bf16 each.
template <int JT>
struct Frags {
  bf16x8_t a[4], b[JT];
};

// Scheduling hint for one k step: its LDS fragment reads go out two per MFMA
// at the front, so each has at least the remaining MFMAs of the step to land.
template <int kReads, int kMfma>
__device__ __forceinline__ void schedule_reads_front() {
  constexpr int kGroups = (kReads + 1) / 2;
#pragma unroll
  for (int q = 0; q < kGroups; ++q) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // two LDS reads
  }
  __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kGroups, 0);
}

// Ring of P part slots.  A stage (BK deep) has two parts, its W rows and its
// X rows; part 2s + 0 / 2s + 1 (W / X of stage s) lives in slot (2s + o) % P.
// Within a stage the wave runs kSub k steps, each reading the next step's
// fragments while its MFMAs run.  Before the last k step every wave waits for
// its own fragment reads (so stage s is no longer read) and for stage s + 1 to
// have landed, then one barrier; after it the two freed slots take parts
// 2s + P and 2s + P + 1.  With P odd the W part of a stage is issued one stage
// before its X part, and about (P - 2) / 2 stages of loads are in flight
// while a stage is consumed.
template <int P, int BK, bool SPLIT>
__global__ __launch_bounds__(kWaves * 64, 2) void entropy_gemm_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, int n_tok, int d, int V, int n_vsplit,
    int n_vt, int n_tt, float* __restrict__ part_m, float* __restrict__ part_s, float* __restrict__ part_t) {
  using G = Geom<BK>;
  constexpr int JT = G::JT;
  static_assert(kBV == kBT, "W and X parts share one slot size");
  static_assert(P >= 4, "the ring needs at least two stages");
  static_assert(G::kSub >= 2, "the barrier sits between the last two k steps of a stage");
  static_assert(G::kInstW == G::kInstX, "equal load counts per part");
  static_assert(4 * G::JT >= 2 * G::kInstW, "one transfer per MFMA of a k step");
  constexpr int L = G::kInstW;  // vector-memory instructions per wave per part
  __shared__ __attribute__((aligned(16))) char lds[P * G::kPartBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave & 1;   // which 128-row half of the vocabulary tile
  const int wt = wave >> 1;  // which TW-token slice of the token tile

  // ---- workgroup -> (vocabulary slice, token tile)
  int vs, tt;
  {
    const int bid = blockIdx.x;
    constexpr int R = 32;  // workgroups resident on one XCD
    if (n_vsplit == 16 && (n_tt % (R / 2)) == 0) {
      const int xcd = bid & 7, j = bid >> 3;
      const int wave_idx = j / R, jj = j % R;
      vs = (jj & 3) * 4 + (xcd & 3);
      tt = wave_idx * (R / 2) + (xcd >> 2) * (R / 4) + (jj >> 2);
    } else {
      vs = bid % n_vsplit;
      tt = bid / n_vsplit;
    }
  }
  const int nk = d / BK;
  const int n_my_tiles = (n_vt - vs + n_vsplit - 1) / n_vsplit;
  const size_t row_stride = size_t(d) * 2;  // bytes per row of W and X

  // ---- staging: lane l of instruction i fills row kRowsPerInst*(kWaves i + wave) + l / kChunks,
  // physical chunk l % kChunks, i.e. logical chunk swz(row, l % kChunks) of that row.
  int st_row[G::kInstW];
  uint32_t st_chunk_off[G::kInstW], offx[G::kInstX];
  const char* xt = reinterpret_cast<const char*>(X) + size_t(tt) * kBT * row_stride;
#pragma unroll
  for (int i = 0; i < G::kInstW; ++i) {
    st_row[i] = G::kRowsPerInst * (kWaves * i + wave) + lane / G::kChunks;
    st_chunk_off[i] = uint32_t(G::swz(st_row[i], lane % G::kChunks) * 16);
  }
#pragma unroll
  for (int i = 0; i < G::kInstX; ++i) {
    const int tr = min(tt * kBT + st_row[i], n_tok - 1) - tt * kBT;
    offx[i] = uint32_t(tr) * uint32_t(row_stride) + st_chunk_off[i];
  }

  // ---- prefetch of parts in order 0, 1, 2, ...: part q is operand q % 2 of
  // stage q / 2 = (tile, ks).  Parts past the end re-load the last stage into
  // the slot being freed (never read), so every barrier issues exactly 2 L
  // loads per wave and the waits below are the same on every stage; the loop
  // body stays one basic block.
  int pf_tile = 0, pf_ks = 0, pf_slot = 0, pf_op = 0;
  // Source and destination of the next part; advances the part counters.
  struct Part {
    const char* src;  // W: start of the vocabulary tile's rows at depth ks; X: same for the token tile
    char* dst;        // this wave's first 1 KB block of the slot
    int vt;           // vocabulary tile (W parts)
  };
  auto next_part = [&](int op) {
    const bool live = pf_tile < n_my_tiles;
    const int ks = live ? pf_ks : nk - 1;
    Part p;
    p.dst = lds + pf_slot * G::kPartBytes + G::kRowsPerInst * wave * G::kRowBytes;
    p.vt = vs + (live ? pf_tile : n_my_tiles - 1) * n_vsplit;
    if (op == 0) {
      p.src = reinterpret_cast<const char*>(W) + size_t(p.vt) * kBV * row_stride + size_t(ks) * G::kRowBytes;
    } else {
      p.src = xt + size_t(ks) * G::kRowBytes;
      const bool wrap = pf_ks + 1 == nk;
      pf_ks = wrap ? 0 : pf_ks + 1;
      pf_tile = wrap ? pf_tile + 1 : pf_tile;
    }
    pf_slot = pf_slot + 1 == P ? 0 : pf_slot + 1;
    return p;
  };
  // Transfer i (of L) of a part: 1 KB, kRowsPerInst rows.
  auto dma_one = [&](const Part& p, int op, int i) {
    char* dst = p.dst + G::kRowsPerInst * kWaves * i * G::kRowBytes;
    if (op == 0) {
      const int vr = min(p.vt * kBV + st_row[i], V - 1) - p.vt * kBV;
      lds_dma16(p.src + (uint32_t(vr) * uint32_t(row_stride) + st_chunk_off[i]), dst);
    } else {
      lds_dma16(p.src + offx[i], dst);
    }
  };
  auto issue_part = [&]() {
    const int op = pf_op;
    const Part p = next_part(op);
#pragma unroll
    for (int i = 0; i < L; ++i) dma_one(p, op, i);
    pf_op ^= 1;
  };
  // The two parts issued at every barrier: their operands are fixed, since an
  // even number of parts precedes each barrier's pair.
  constexpr int kOpA = P % 2, kOpB = kOpA ^ 1;

  // ---- fragment reads: lane (row r = lane % 32, half h = lane / 32) reads 8 bf16 at
  // k offset 16 kk + 8 h of row r of each 32-row block.
  const int frag_row = lane & 31;
  const int frag_half = lane >> 5;
  uint32_t fa_off[G::kSub][4], fb_off[G::kSub][JT];  // byte offsets inside a stage, per k step
#pragma unroll
  for (int kk = 0; kk < G::kSub; ++kk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ra = wv * 128 + i * 32 + frag_row;
      fa_off[kk][i] = ra * G::kRowBytes + G::swz(ra, kk * 2 + frag_half) * 16;
    }
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int rb = wt * G::TW + j * 32 + frag_row;
      fb_off[kk][j] = rb * G::kRowBytes + G::swz(rb, kk * 2 + frag_half) * 16;
    }
  }
  auto read_frags = [&](Frags<JT>& f, int slot_w, int slot_x, int kk) {
    const char* bw = lds + slot_w * G::kPartBytes;
    const char* bx = lds + slot_x * G::kPartBytes;
#pragma unroll
    for (int i = 0; i < 4; ++i) f.a[i] = *reinterpret_cast<const bf16x8_t*>(bw + fa_off[kk][i]);
#pragma unroll
    for (int j = 0; j < JT; ++j) f.b[j] = *reinterpret_cast<const bf16x8_t*>(bx + fb_off[kk][j]);
  };
  constexpr int kReads = 4 + JT;       // LDS reads per k step
  constexpr int kMfma = 4 * JT;        // MFMAs per k step

  // ---- per-lane entropy state for the JT token columns this lane owns
  Ent2 st[JT];
#pragma unroll
  for (int cb = 0; cb < JT; ++cb) st[cb] = Ent2{-INFINITY, 0.f, 0.f};

  // ---- prologue: the first parts in flight; wait for stage 0, read its first fragments
  constexpr int kPrologue = SPLIT ? P - 1 : P;
#pragma unroll
  for (int q = 0; q < kPrologue; ++q) issue_part();
  wait_vm<(kPrologue - 2) * L>();
  lds_barrier();
  Frags<JT> f[2];
  read_frags(f[0], 0, 1, 0);
  int sw = 0;  // slot of the W part of the current stage; its X part is in sw + 1 (mod P)

  // MFMAs of one k step with the L transfers of part p0 and then, if n1 > 0,
  // those of part p1 threaded between them, one per MFMA, so a burst of
  // transfers never holds the wave away from the matrix core.
  auto mfma_with_dma = [&](f32x16_t(&acc)[4][JT], const Frags<JT>& cur, const Part& p0, int op0, const Part& p1,
                           int op1, int n1) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < JT; ++j) {
        const int m = i * JT + j;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.a[i], cur.b[j], acc[i][j], 0, 0, 0);
        if (m < L)
          dma_one(p0, op0, m);
        else if (m < L + n1)
          dma_one(p1, op1, m - L);
        __builtin_amdgcn_sched_barrier(0);
      }
  };

  for (int tile = 0; tile < n_my_tiles; ++tile) {
    f32x16_t acc[4][JT];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < JT; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    for (int ks = 0; ks < nk; ++ks) {
      const int sx = sw + 1 == P ? 0 : sw + 1;
      const int sw_next = sx + 1 == P ? 0 : sx + 1;
      const int sx_next = sw_next + 1 == P ? 0 : sw_next + 1;
#pragma unroll
      for (int u = 0; u < G::kSub; ++u) {
        Frags<JT>& cur = f[u & 1];
        Frags<JT>& nxt = f[(u + 1) & 1];
        if (u + 1 < G::kSub) {
          read_frags(nxt, sw, sx, u + 1);
          if (SPLIT && u == 0) {
            // the second part freed at the previous barrier goes out here
            const Part pb = next_part(kOpB);
            mfma_with_dma(acc, cur, pb, kOpB, pb, kOpB, 0);
            continue;
          }
        } else {
          // This wave's reads of the stage are done (lgkmcnt 0 inside the
          // barrier) and the next stage has landed (only the P - 4 parts
          // issued after it may still be in flight): after the barrier nobody
          // reads this stage's slots again, so they take the next two parts.
          // The previous k step's MFMAs stay in front of the wait.
          __builtin_amdgcn_sched_barrier(0);
          wait_vm<(P - 4) * L>();
          lds_barrier();
          const Part pa = next_part(kOpA);
          if (SPLIT) {
            read_frags(nxt, sw_next, sx_next, 0);  // past the last stage: read and never used
            mfma_with_dma(acc, cur, pa, kOpA, pa, kOpA, 0);
          } else {
            const Part pb = next_part(kOpB);
            read_frags(nxt, sw_next, sx_next, 0);  // past the last stage: read and never used
            mfma_with_dma(acc, cur, pa, kOpA, pb, kOpB, L);
          }
          continue;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < JT; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.a[i], cur.b[j], acc[i][j], 0, 0, 0);
        schedule_reads_front<kReads, kMfma>();
      }
      sw = sw_next;
    }

    // ---- fold the finished tile into the running states.  acc[i][j][r] is the
    // logit of vocabulary row vt*256 + wv*128 + i*32 + 8*(r/4) + 4*frag_half + r%4
    // for token tt*BT + wt*TW + j*32 + frag_row.
    //
    // The state (m, s, t) is kept relative to a reference m that is the running
    // log-sum-exp after each tile (rebased so that s = 1).  Full tiles are then
    // folded with 3 VALU ops and one exp2 per logit and no max pass; a tile whose
    // logits exceed the reference by more than 2^64 in weight (or overflow) is
    // refolded exactly with its own max.  The ragged last vocabulary tile always
    // takes the exact, masked path.
    const int vt = vs + tile * n_vsplit;
    const bool ragged = (vt + 1) * kBV > V;
    const int lim = V - (vt * kBV + wv * 128 + 4 * frag_half);  // live rows: offset < lim
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      Ent2 e = st[j];
      bool exact = ragged;
      if (!ragged) {
        if (tile == 0) {  // first tile: the tile's own max is the reference
          float mx = acc[0][j][0];
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, acc[i][j][r]);
          e = Ent2{mx * kLog2e, 0.f, 0.f};
        }
        float s = e.s, t = e.t;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float dd = fmaf(acc[i][j][r], kLog2e, -e.m);
            const float p = fast_exp2(dd);
            s += p;
            t = fmaf(p, dd, t);
          }
          __builtin_amdgcn_sched_barrier(0);  // block by block: bounds live copies
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
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const bool live = !ragged || i * 32 + 8 * (r >> 2) + (r & 3) < lim;
            mx = live ? fmaxf(mx, acc[i][j][r]) : mx;
          }
        const float mnew = fmaxf(e.m, mx * kLog2e);
        const float dl = fmaxf(e.m - mnew, kExp2Floor);
        const float f = fast_exp2(dl);
        float s = f * e.s;
        float t = f * (e.t + e.s * dl);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            // dead rows enter as -inf: dd clamps to the floor and adds 0 * floor,
            // also while mnew is still -inf (a lane with no live row yet)
            const bool live = !ragged || i * 32 + 8 * (r >> 2) + (r & 3) < lim;
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
  }  // tile

  // ---- lanes l and l+32 hold the same tokens: merge them
#pragma unroll
  for (int j = 0; j < JT; ++j) {
    Ent2 o;
    o.m = __shfl_xor(st[j].m, 32, 64);
    o.s = __shfl_xor(st[j].s, 32, 64);
    o.t = __shfl_xor(st[j].t, 32, 64);
    st[j] = ent2_merge(st[j], o);
  }
  // ---- the two vocabulary halves (wv = 0, 1) hold the same tokens: merge through LDS
  __syncthreads();  // every wave is done with the ring (no loads remain in flight)
  float* xbuf = reinterpret_cast<float*>(lds);  // [BT tokens][3]
  if (wv == 1 && frag_half == 0) {
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      float* p = xbuf + (wt * G::TW + j * 32 + frag_row) * 3;
      p[0] = st[j].m;
      p[1] = st[j].s;
      p[2] = st[j].t;
    }
  }
  __syncthreads();
  if (wv == 0 && frag_half == 0) {
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int tl = wt * G::TW + j * 32 + frag_row;
      const float* p = xbuf + tl * 3;
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
}

// Merge the n_vsplit partial states of each token and write H in nats:
// H = ln2 * (log2 s - t / s).
__global__ __launch_bounds__(256) void entropy_merge_kernel(const float* __restrict__ part_m,
                                                            const float* __restrict__ part_s,
                                                            const float* __restrict__ part_t, int n_tok,
                                                            int n_vsplit, float* __restrict__ H) {
  const int tok = blockIdx.x * 256 + threadIdx.x;
  if (tok >= n_tok) return;
  Ent2 a{part_m[tok], part_s[tok], part_t[tok]};
  for (int v = 1; v < n_vsplit; ++v) {
    const size_t o = size_t(v) * n_tok + tok;
    a = ent2_merge(a, Ent2{part_m[o], part_s[o], part_t[o]});
  }
  H[tok] = kLn2 * (fast_log2(a.s) - a.t / a.s);
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
  for (int i = 0; i < 3; ++i) c.take<float>(size_t(choose_vsplit(n_vt)) * n_tok);
  return c.bytes();
}

extern "C" int estp_token_entropy(const void* X, const void* W, int64_t n_tok, int32_t d, int32_t V, int dtype,
                                  float* H, void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  ESTP_REQUIRE(X && W && H, ESTP_ERR_INVALID_ARG, "estp_token_entropy: X, W and H must be non-null");
  ESTP_REQUIRE(n_tok >= 1 && n_tok <= INT32_MAX, ESTP_ERR_INVALID_ARG,
               "estp_token_entropy: n_tok must be in [1, 2^31), got %lld", (long long)n_tok);
  ESTP_REQUIRE(V >= 1, ESTP_ERR_INVALID_ARG, "estp_token_entropy: V must be >= 1, got %d", V);
  ESTP_REQUIRE(d >= 8 && d % 8 == 0, ESTP_ERR_INVALID_ARG,
               "estp_token_entropy: d must be a positive multiple of 8, got %d", d);
  ESTP_REQUIRE(dtype == ESTP_BF16 || dtype == ESTP_F32, ESTP_ERR_INVALID_ARG,
               "estp_token_entropy: unknown dtype %d", dtype);
  ESTP_REQUIRE(dtype == ESTP_BF16, ESTP_ERR_UNSUPPORTED, "estp_token_entropy: only ESTP_BF16 inputs are supported");
  ESTP_REQUIRE(d % 32 == 0, ESTP_ERR_UNSUPPORTED,
               "estp_token_entropy: d must be a multiple of 32 for the matrix-core path, got %d", d);
  ESTP_REQUIRE(size_t(d) * 2 * kBV < (size_t(1) << 32), ESTP_ERR_UNSUPPORTED,
               "estp_token_entropy: d = %d too large", d);
  ESTP_REQUIRE(aligned(X, 16) && aligned(W, 16), ESTP_ERR_INVALID_ARG,
               "estp_token_entropy: X and W must be 16-byte aligned");
  const size_t need = estp_token_entropy_workspace_size(n_tok, d, V, dtype);
  ESTP_REQUIRE(workspace_bytes >= need, ESTP_ERR_WORKSPACE,
               "estp_token_entropy: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  ESTP_REQUIRE(workspace && aligned(workspace, 256), ESTP_ERR_INVALID_ARG,
               "estp_token_entropy: workspace must be non-null and 256-byte aligned");

  const int n = int(n_tok);
  const int n_vt = (V + kBV - 1) / kBV;
  const int n_tt = (n + kBT - 1) / kBT;
  const int n_vsplit = choose_vsplit(n_vt);
  Carver c(workspace);
  float* pm = c.take<float>(size_t(n_vsplit) * n);
  float* ps = c.take<float>(size_t(n_vsplit) * n);
  float* pt = c.take<float>(size_t(n_vsplit) * n);
  hipStream_t s = static_cast<hipStream_t>(stream);

  const dim3 grid(n_vsplit * n_tt), block(kWaves * 64);
  const uint16_t* Xh = static_cast<const uint16_t*>(X);
  const uint16_t* Wh = static_cast<const uint16_t*>(W);
  if (d % 64 == 0)
    entropy_gemm_kernel<5, 64, false><<<grid, block, 0, s>>>(Xh, Wh, n, int(d), int(V), n_vsplit, n_vt, n_tt, pm, ps, pt);
  else
    entropy_gemm_kernel<7, 32, false><<<grid, block, 0, s>>>(Xh, Wh, n, int(d), int(V), n_vsplit, n_vt, n_tt, pm, ps, pt);
  ESTP_CHECK_LAUNCH("entropy_gemm_kernel");
  entropy_merge_kernel<<<dim3((n + 255) / 256), dim3(256), 0, s>>>(pm, ps, pt, n, n_vsplit, H);
  ESTP_CHECK_LAUNCH("entropy_merge_kernel");
  return ESTP_OK;
}
