// Token entropy (Eq. 2) for fp32 hidden states and LM-head weights, with fp32
// arithmetic throughout.
//
// A workgroup of 256 threads owns one 128-token tile and, in turn, the
// 128-row vocabulary tiles of one vocabulary slice (tiles slice,
// slice + n_vsplit, ...).  Each thread accumulates an 8 x 8 block of logits
// (vocabulary rows 4 rv .. 4 rv + 3 and 64 + 4 rv .. + 3, tokens 4 ct .. + 3 and
// 64 + 4 ct .. + 3) from 32-deep k stages of W and X held k-major in LDS: a
// thread reads two float4 of each operand per k and issues 64 FMAs.  The next
// stage is loaded into registers while the current one is multiplied, and
// written to the other LDS buffer afterwards (one barrier per stage).  After
// the last stage of a vocabulary tile a thread folds its logits into one
// online-softmax state per token column (Ent2, base 2; exact, with the tile's
// own max).  At the end the 16 threads that share a token column merge their
// states (two lane exchanges, then the four waves through LDS, in a fixed
// order) and the slice writes the partial layout that entropy_merge_kernel
// reduces.  The kArg variant also keeps each token column's largest logit and
// its lowest vocabulary index through the same merges.
#include "estp_common.h"
#include "f32_paths.h"

namespace estp {
namespace detail {
namespace {

constexpr int kFV = 128;        // vocabulary rows per tile
constexpr int kFT = 128;        // tokens per tile
constexpr int kFK = 32;         // k depth of one stage
constexpr int kFPitch = 132;    // LDS row pitch (floats) of a k-major tile; keeps float4 alignment
constexpr int kFThreads = 256;
constexpr int kFLoads = kFV * kFK / 4 / kFThreads;  // float4 loads per thread, operand and stage
static_assert(kFV == kFT && kFLoads == 4, "one load pattern serves both operands");
static_assert(kFPitch % 4 == 0 && kFPitch >= kFV, "pitch");

}  // namespace

// b replaces a when larger, or equal with a lower index.
__device__ __forceinline__ void arg_merge_f32(float& av, int& ai, float bv, int bi) {
  const bool take = bv > av || (bv == av && bi < ai);
  av = take ? bv : av;
  ai = take ? bi : ai;
}

template <bool kArg>
__global__ __launch_bounds__(kFThreads) void entropy_f32_kernel(const float* __restrict__ X,
                                                                const float* __restrict__ W, int n_tok, int d,
                                                                int V, int n_vsplit, int n_vt,
                                                                float* __restrict__ part_m,
                                                                float* __restrict__ part_s,
                                                                float* __restrict__ part_t,
                                                                float* __restrict__ part_zmax,
                                                                int* __restrict__ part_arg) {
  __shared__ __attribute__((aligned(16))) float ws[2][kFK][kFPitch];
  __shared__ __attribute__((aligned(16))) float xs[2][kFK][kFPitch];
  const int tid = threadIdx.x;
  const int slice = blockIdx.x % n_vsplit;
  const int t0 = (blockIdx.x / n_vsplit) * kFT;
  const int rv = tid >> 4, ct = tid & 15;
  const int n_k = (d + kFK - 1) / kFK;
  const int n_mine = (n_vt - slice + n_vsplit - 1) / n_vsplit;  // vocabulary tiles of this slice
  const int n_steps = n_mine * n_k;

  // float4 i of a thread: row (tid + 256 i) / 8 of the tile, k offset 4 ((tid + 256 i) % 8); eight
  // threads cover one 128-byte run of a row.  Rows past V or n_tok and k past d read as zero.
  float4 rw[kFLoads], rx[kFLoads];
  auto load = [&](int step) {
    const int v0 = (slice + (step / n_k) * n_vsplit) * kFV;
    const int k0 = (step % n_k) * kFK;
#pragma unroll
    for (int i = 0; i < kFLoads; ++i) {
      const int idx = tid + kFThreads * i;
      const int r = idx >> 3, k = k0 + 4 * (idx & 7);
      const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
      rw[i] = (v0 + r < V && k < d) ? *reinterpret_cast<const float4*>(W + size_t(v0 + r) * d + k) : z;
      rx[i] = (t0 + r < n_tok && k < d) ? *reinterpret_cast<const float4*>(X + size_t(t0 + r) * d + k) : z;
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kFLoads; ++i) {
      const int idx = tid + kFThreads * i;
      const int r = idx >> 3, k = 4 * (idx & 7);
      ws[buf][k][r] = rw[i].x;
      ws[buf][k + 1][r] = rw[i].y;
      ws[buf][k + 2][r] = rw[i].z;
      ws[buf][k + 3][r] = rw[i].w;
      xs[buf][k][r] = rx[i].x;
      xs[buf][k + 1][r] = rx[i].y;
      xs[buf][k + 2][r] = rx[i].z;
      xs[buf][k + 3][r] = rx[i].w;
    }
  };

  float acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  Ent2 st[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) st[j] = Ent2{-INFINITY, 0.f, 0.f};
  float zmax[8];  // kArg: largest logit per token column and its vocabulary index
  int zarg[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    zmax[j] = -INFINITY;
    zarg[j] = INT32_MAX;
  }

  load(0);
  store(0);
  __syncthreads();
  for (int step = 0; step < n_steps; ++step) {
    const int buf = step & 1;
    const bool more = step + 1 < n_steps;
    if (more) load(step + 1);
#pragma unroll 4
    for (int k = 0; k < kFK; ++k) {
      const float4 a0 = *reinterpret_cast<const float4*>(&ws[buf][k][4 * rv]);
      const float4 a1 = *reinterpret_cast<const float4*>(&ws[buf][k][64 + 4 * rv]);
      const float4 b0 = *reinterpret_cast<const float4*>(&xs[buf][k][4 * ct]);
      const float4 b1 = *reinterpret_cast<const float4*>(&xs[buf][k][64 + 4 * ct]);
      const float a[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      const float b[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    if ((step + 1) % n_k == 0) {
      // last stage of vocabulary tile vt: fold its logits, rows past V left out
      const int v0 = (slice + (step / n_k) * n_vsplit) * kFV;
      bool valid[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) valid[i] = v0 + (i < 4 ? 4 * rv + i : 64 + 4 * rv + i - 4) < V;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float mx = -INFINITY;
        int imx = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          // rows ascend with i: a strict compare keeps the lowest index among equal logits
          const bool up = valid[i] && acc[i][j] > mx;
          imx = up ? i : imx;
          mx = up ? acc[i][j] : mx;
        }
        if (kArg && mx > zmax[j]) {
          zmax[j] = mx;
          zarg[j] = v0 + (imx < 4 ? 4 * rv + imx : 64 + 4 * rv + imx - 4);
        }
        if (valid[0]) {  // row 4 rv of the tile is the thread's first; none valid -> nothing to add
          const float m2 = mx * kLog2e;
          float s = 0.f, t = 0.f;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            if (!valid[i]) continue;
            const float z = fmaf(acc[i][j], kLog2e, -m2);
            const float p = fast_exp2(z);
            s += p;
            t = fmaf(p, z, t);
          }
          st[j] = ent2_merge(st[j], Ent2{m2, s, t});
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i][j] = 0.f;
      }
    }
    if (more) store(buf ^ 1);
    __syncthreads();
  }

  // threads tid, tid ^ 16, tid ^ 32 (same wave) share their token columns ...
#pragma unroll
  for (int j = 0; j < 8; ++j) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const Ent2 other{__shfl_xor(st[j].m, o, 64), __shfl_xor(st[j].s, o, 64), __shfl_xor(st[j].t, o, 64)};
      st[j] = ent2_merge(st[j], other);
      if (kArg) arg_merge_f32(zmax[j], zarg[j], __shfl_xor(zmax[j], o, 64), __shfl_xor(zarg[j], o, 64));
    }
  }
  // ... and so do the four waves: merged through LDS (the stage buffers are free after the last barrier)
  float* red = &ws[0][0][0];  // [3 (5 with kArg)][4 waves][128 tokens]
  static_assert(5 * 4 * kFT <= 2 * kFK * kFPitch, "exchange fits in the stage buffer");
  const int wave = tid >> 6, lane = tid & 63;
  if (lane < 16) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int col = j < 4 ? 4 * ct + j : 64 + 4 * ct + j - 4;
      red[(0 * 4 + wave) * kFT + col] = st[j].m;
      red[(1 * 4 + wave) * kFT + col] = st[j].s;
      red[(2 * 4 + wave) * kFT + col] = st[j].t;
      if (kArg) {
        red[(3 * 4 + wave) * kFT + col] = zmax[j];
        red[(4 * 4 + wave) * kFT + col] = __int_as_float(zarg[j]);
      }
    }
  }
  __syncthreads();
  if (tid < kFT && t0 + tid < n_tok) {
    Ent2 a{red[tid], red[4 * kFT + tid], red[8 * kFT + tid]};
    for (int w = 1; w < 4; ++w) a = ent2_merge(a, Ent2{red[w * kFT + tid], red[(4 + w) * kFT + tid],
                                                       red[(8 + w) * kFT + tid]});
    const size_t o = size_t(slice) * n_tok + t0 + tid;
    part_m[o] = a.m;
    part_s[o] = a.s;
    part_t[o] = a.t;
    if (kArg) {
      float zb = red[12 * kFT + tid];
      int ib = __float_as_int(red[16 * kFT + tid]);
      for (int w = 1; w < 4; ++w) arg_merge_f32(zb, ib, red[(12 + w) * kFT + tid], __float_as_int(red[(16 + w) * kFT + tid]));
      part_zmax[o] = zb;
      part_arg[o] = ib;
    }
  }
}

size_t entropy_f32_workgroups(int n_tok, int n_vsplit) {
  return size_t(n_vsplit) * size_t((n_tok + kFT - 1) / kFT);
}

void launch_entropy_f32(const float* X, const float* W, int n_tok, int d, int V, int n_vsplit, float* part_m,
                        float* part_s, float* part_t, float* part_zmax, int* part_arg, hipStream_t s) {
  const int n_vt = (V + kFV - 1) / kFV;
  const int n_tt = (n_tok + kFT - 1) / kFT;
  const dim3 grid(n_vsplit * n_tt), block(kFThreads);
  if (part_arg)
    entropy_f32_kernel<true><<<grid, block, 0, s>>>(X, W, n_tok, d, V, n_vsplit, n_vt, part_m, part_s, part_t,
                                                    part_zmax, part_arg);
  else
    entropy_f32_kernel<false><<<grid, block, 0, s>>>(X, W, n_tok, d, V, n_vsplit, n_vt, part_m, part_s, part_t,
                                                     nullptr, nullptr);
}

}  // namespace detail
}  // namespace estp
