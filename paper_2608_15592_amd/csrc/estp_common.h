// Shared helpers of libestp: bf16 handling, exp2/log2, wave reductions, the
// per-thread error message and workspace carving.  gfx950 (CDNA4) only:
// wave64, matrix-core (MFMA) bf16 instructions with fp32 accumulation.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include <vector>

#include "estp.h"

namespace estp {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) void* lds_ptr_t;
// Generic pointer into __shared__ memory -> LDS address-space pointer.
__device__ __forceinline__ lds_ptr_t to_lds(void* p) { return (lds_ptr_t)(p); }

// 16-byte global -> LDS transfer (global_load_lds_dwordx4): each lane of the
// wave fetches 16 bytes from its own `src`; they land in LDS at
// dst_wave_base + 16 * lane.  `dst_wave_base` must be uniform across the wave.
// The builtin only exists in the device pass; the host pass (which only needs
// the kernel's launch stub) sees an empty body.
__device__ __forceinline__ void lds_dma16(const void* src, void* dst_wave_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(src, to_lds(dst_wave_base), 16, 0, 0);
#endif
}

// Buffer resource (V#) over `bytes` bytes from `base`: raw dword addressing
// (stride 0); a lane whose byte offset is at or past `bytes` reads zero and
// touches no memory.  Word 3 is the gfx9 data-format word for dword access.
typedef __amdgpu_buffer_rsrc_t buf_rsrc_t;
__device__ __forceinline__ buf_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, int(bytes), 0x00020000);
}

// 16-byte buffer -> LDS transfer (buffer_load_dwordx4 ... lds): lane l reads
// the 16 bytes at voffset(l) + soffset of the resource; they land in LDS at
// dst_wave_base + 16 * l.  `soffset` and `dst_wave_base` must be uniform.
__device__ __forceinline__ void lds_dma16_buf(buf_rsrc_t r, uint32_t voffset, uint32_t soffset,
                                              void* dst_wave_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, to_lds(dst_wave_base), 16, voffset, soffset, 0, 0);
#endif
}

// s_waitcnt vmcnt(N): wait until at most N of this wave's vector-memory
// operations are outstanding (they retire in issue order), including global ->
// LDS transfers; other counters untouched.  gfx9 encoding: vmcnt[3:0] |
// expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at bits [15:14].
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x0F70);
}

// Workgroup barrier that leaves outstanding global loads in flight (unlike
// __syncthreads, whose fence drains them): waits only for this wave's LDS
// operations, then s_barrier.  The signal fences keep the compiler from moving
// memory accesses across it.  Visibility of global -> LDS transfers is the
// caller's job (wait_vm before the barrier).
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Barrier for a ring whose slots are only ever written by global -> LDS
// transfers: no LDS wait at all.  Safe when every LDS read of the slot that is
// refilled after this barrier has already been consumed (its data used) by the
// reading wave before the barrier.
__device__ __forceinline__ void ring_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// exp2 of anything below this is 0 in fp32; used to clamp (-inf) - (-inf) style cases.
constexpr float kExp2Floor = -256.0f;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// v_exp_f32 / v_log_f32: hardware base-2 exponential and logarithm.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Online-softmax state in base-2 units: m = running max of z*log2e,
// s = sum 2^(z2 - m), t = sum 2^(z2 - m) * (z2 - m).
struct Ent2 {
  float m, s, t;
};

// Merge two states; exp2 arguments are clamped so -inf maxima (empty states)
// contribute exactly nothing instead of NaN.
__device__ __forceinline__ Ent2 ent2_merge(Ent2 a, Ent2 b) {
  float M = fmaxf(a.m, b.m);
  float da = fmaxf(a.m - M, kExp2Floor);
  float db = fmaxf(b.m - M, kExp2Floor);
  float fa = fast_exp2(da), fb = fast_exp2(db);
  Ent2 r;
  r.m = M;
  r.s = fa * a.s + fb * b.s;
  r.t = fa * (a.t + a.s * da) + fb * (b.t + b.s * db);
  return r;
}

// ------------------------------------------------------------------ host side

void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

// Debug mode: ESTP_DEBUG_CHECKS=1 in the environment (read once per process).  Calls that take
// cu_seqlens copy it back and check it before any kernel runs (cu[0] = 0, cu[B] = n_tok, every
// prompt length in [1, max_seqlen]); calls that build a work list on the device copy it back
// and compare it with its definition before the kernels that consume it are launched.  Both
// synchronise the stream, so the mode is for testing, not for graph capture.
bool debug_checks_enabled();
// n_tok < 0: the call does not state n_tok, cu_seqlens[B] is not compared.
int debug_check_cu(const char* fn, const int32_t* cu_dev, int32_t B, int64_t n_tok, int32_t max_seqlen,
                   hipStream_t s, std::vector<int>* cu_out);
int debug_check_list(const char* fn, const int2* list_dev, const std::vector<int2>& expect, hipStream_t s);

// Compute units of the current device (cached per device; 0 when the runtime cannot tell).
constexpr int kMaxDevices = 64;
int current_device_cu_count();

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// A launch covers at most 2^32 - 1 work-items along its x dimension.
inline bool fits_launch(size_t workgroups, size_t threads) {
  return workgroups >= 1 && workgroups <= size_t(UINT32_MAX) / threads;
}

// Sequential carving of a caller workspace into 256-byte aligned pieces.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* p) : base(static_cast<char*>(p)) {}
  template <typename T>
  T* take(size_t count) {
    off = align_up(off, 256);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t bytes() const { return align_up(off, 256); }
};

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace estp

#define ESTP_REQUIRE(cond, code, ...)  \
  do {                                 \
    if (!(cond)) {                     \
      ::estp::set_error(__VA_ARGS__);  \
      return (code);                   \
    }                                  \
  } while (0)

#define ESTP_CHECK_LAUNCH(what)                                                          \
  do {                                                                                   \
    hipError_t e_ = hipGetLastError();                                                   \
    if (e_ != hipSuccess) {                                                              \
      ::estp::set_error("%s: %s", (what), hipGetErrorString(e_));                        \
      return ESTP_ERR_HIP;                                                               \
    }                                                                                    \
  } while (0)
