// Launchers of the fp32-input kernels (entropy_f32.hip, importance_f32.hip).
// On gfx950 the fp32 vector FMA rate equals the fp32 matrix-core rate (both
// 157.3 TFLOP/s dense), so these contractions are register-tiled VALU code;
// the bf16 calls keep the matrix-core kernels.  Both write the same
// intermediate layouts as the bf16 kernels, so the merge and reduce kernels
// are shared.
#pragma once

#include <hip/hip_runtime.h>

namespace estp {
namespace detail {

// Workgroups in launch_entropy_f32's grid.
size_t entropy_f32_workgroups(int n_tok, int n_vsplit);
// Per-slice online-softmax partial states (part_m/s/t [n_vsplit, n_tok], base
// 2) of the logits W x for every token; 1 <= n_vsplit <= ceil(V / 128).  With
// part_arg non-null, also each slice's largest logit (part_zmax) and its
// lowest vocabulary index (part_arg), same layout.
void launch_entropy_f32(const float* X, const float* W, int n_tok, int d, int V, int n_vsplit, float* part_m,
                        float* part_s, float* part_t, float* part_zmax, int* part_arg, hipStream_t s);

// The two importance passes over the same grid as the bf16 kernels: n_rows
// 256-row block entries (from `blist`, n_bound entries, when non-null; else the
// nqb x B longest-prompt grid) times L * Hq (pass 1) or L * Hkv (pass 2).
// Pass 1 runs when run_lse is set and writes lse2 [L, Hq, n_tok] in base 2;
// pass 2 reads lse2 scaled by lse_mul and writes the column masses part
// [L, Hkv, n_tok].
void launch_importance_f32(int dh, const float* Q, const float* K, const int* cu, int B, int n_tok, int L, int Hq,
                           int Hkv, int nqb, float c2, const int2* blist, size_t n_rows, int n_bound, bool run_lse,
                           float* lse2, float lse_mul, int strict, float* part, hipStream_t s);

}  // namespace detail
}  // namespace estp
