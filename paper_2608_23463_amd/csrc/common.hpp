// Device-side building blocks shared by every kernel of the library:
// element types, 16-byte vector access, fp32<->bf16 conversion and the
// MFMA fragment abstraction for gfx950 (CDNA4, 64-wide wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pf {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;  // MI355X: 8 accelerator complex dies, workgroups dealt round-robin

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }  // round to nearest even

template <typename T>
__device__ __forceinline__ float load_f32(const T* p, int64_t i) {
  return p ? to_f32(p[i]) : 0.0f;
}

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

// Raw buffer access (gfx9 descriptor word 3 = 0x00020000). A load whose byte
// offset plus size exceeds `bytes` returns zero, so tile edges need no
// branches; kOOB is an offset that is always out of range.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}
// Same descriptor, with base and size forced into scalar registers (they are
// uniform across the wave; this keeps the compiler from looping over lanes).
__device__ __forceinline__ rsrc_t make_rsrc_uniform(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  return make_rsrc(reinterpret_cast<const void*>(((uint64_t)hi << 32) | lo), __builtin_amdgcn_readfirstlane(bytes));
}
__device__ __forceinline__ u32x4 buf_ld16(rsrc_t r, uint32_t voff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0);
}
// Direct global -> LDS load of 16 bytes per lane: lane l of the wave writes
// lds_base + 16 * l (out-of-range lanes write zeros). lds_base is wave-uniform.
__device__ __forceinline__ void buf_ld16_lds(rsrc_t r, uint32_t voff, void* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_base, 16, voff, 0, 0, 0);
}
// The same with a wave-uniform byte offset soff added to every lane's address.
__device__ __forceinline__ void buf_ld16_lds_so(rsrc_t r, uint32_t voff, uint32_t soff, void* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_base, 16, voff, soff, 0, 0);
}
// s_waitcnt immediates (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt in 6:4, lgkmcnt in 11:8); a field at its maximum does not wait.
// Issued through the builtin so the compiler's own wait insertion knows
// about them and does not add redundant waits on younger operations.
constexpr int waitcnt_imm(int vm, int lgkm) { return (vm & 15) | ((vm >> 4) << 14) | (7 << 4) | (lgkm << 8); }
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit counter");
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(N, 15));
}
// Workgroup barrier for LDS hand-offs: this wave's LDS reads have returned
// before any wave passes. Unlike __syncthreads() it does not also wait for
// every outstanding global load (in-flight direct-to-LDS stages stay in
// flight; the caller waits for the stage it needs with wait_vmcnt first).
// The empty asm statements keep the compiler from moving memory accesses
// across the barrier.
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0)); }
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  wait_lgkmcnt0();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// Low part of a two-term bf16 split: v = hi + lo with hi = bf16(v) and
// lo = bf16(v - hi), which together keep ~16 mantissa bits of v. For fp32
// tensors there is no low part.
__device__ __forceinline__ float split_lo(float v) { return (float)(bf16)(v - (float)(bf16)v); }

// Four floats -> four fp8 e5m2 bytes (OCP "bf8" encoding, round to nearest
// even, hardware conversion), saturated to the largest finite +-57344 first;
// byte i holds the i-th value. Normal values span 2^-14 .. 57344.
__device__ __forceinline__ uint32_t pack_bf8x4(float a, float b, float c, float d) {
  auto sat = [](float x) { return fminf(fmaxf(x, -57344.0f), 57344.0f); };
  int w = __builtin_amdgcn_cvt_pk_bf8_f32(sat(a), sat(b), 0, false);
  w = __builtin_amdgcn_cvt_pk_bf8_f32(sat(c), sat(d), w, true);
  return (uint32_t)w;
}

// Eight consecutive elements <-> fp32 (16-byte aligned for bf16, two
// 16-byte accesses for fp32).
__device__ __forceinline__ void load8(const bf16* p, float* v) {
  const bf16x8 x = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)x[i];
}
__device__ __forceinline__ void load8(const float* p, float* v) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p);
  const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i] = a[i];
    v[i + 4] = b[i];
  }
}
// Eight elements held as loaded (not yet widened), so the load can stay in
// flight until raw_to_f32 first needs the values.
template <typename T>
struct Raw8 {
  u32x4 w[sizeof(T) / 2];
};
template <typename T>
__device__ __forceinline__ void raw_load8(const T* p, Raw8<T>& r) {
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 2); ++i) r.w[i] = ld16(reinterpret_cast<const char*>(p) + 16 * i);
}
template <typename T>
__device__ __forceinline__ void raw_to_f32(const Raw8<T>& r, float* v) {
  const T* e = reinterpret_cast<const T*>(r.w);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = to_f32(e[i]);
}
__device__ __forceinline__ void store8(bf16* p, const float* v) {
  bf16x8 x;
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = (bf16)v[i];
  *reinterpret_cast<bf16x8*>(p) = x;
}
__device__ __forceinline__ void store8(float* p, const float* v) {
  f32x4 a, b;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = v[i];
    b[i] = v[i + 4];
  }
  *reinterpret_cast<f32x4*>(p) = a;
  *reinterpret_cast<f32x4*>(p + 4) = b;
}

// Four consecutive elements <-> fp32 (8-byte aligned for bf16, 16 for fp32).
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void load4(const bf16* p, float* v) {
  const bf16x4 x = *reinterpret_cast<const bf16x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (float)x[i];
}
__device__ __forceinline__ void load4(const float* p, float* v) {
  const f32x4 x = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = x[i];
}
__device__ __forceinline__ void store4(bf16* p, const float* v) {
  bf16x4 x;
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = (bf16)v[i];
  *reinterpret_cast<bf16x4*>(p) = x;
}
__device__ __forceinline__ void store4(float* p, const float* v) {
  f32x4 x;
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = v[i];
  *reinterpret_cast<f32x4*>(p) = x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Logistic function on the hardware base-2 exponential and reciprocal (each
// within about one ulp): four VALU operations instead of a full division.
__device__ __forceinline__ float sigmoidf(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-z * 1.4426950408889634f));
}

// ---------------------------------------------------------------------------
// MFMA fragments. One "k16 step" multiplies a 32x16 slice of A by a 16x32
// slice of B into a 32x32 fp32 tile held as 16 floats per lane.
// Lane l supplies row (l % 32) of A / column (l % 32) of B and the eight
// reduction indices (l / 32) * 8 .. +7 of the step. Because A and B use the
// same lane->index assignment, the product is exact regardless of how the
// hardware orders the reduction inside the instruction.
//  bf16: one v_mfma_f32_32x32x16_bf16 (8 bf16 per lane per operand).
//  fp32: eight v_mfma_f32_32x32x2_f32; slot s of lane group g is index g*8+s.
// Output layout of a 32x32 tile: lane l holds column l % 32, register r holds
// row (r / 4) * 8 + (l / 32) * 4 + (r % 4).
// ---------------------------------------------------------------------------
template <typename T>
struct Mma;

template <>
struct Mma<bf16> {
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x16 mma(const frag& a, const frag& b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag load(const bf16* p) {
    return *reinterpret_cast<const frag*>(p);
  }
  static __device__ __forceinline__ frag pack(const float* v) {
    frag f;
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = (bf16)v[i];
    return f;
  }
};

template <>
struct Mma<float> {
  typedef f32x8 frag;
  static __device__ __forceinline__ f32x16 mma(const frag& a, const frag& b, f32x16 c) {
#pragma unroll
    for (int s = 0; s < 8; ++s) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[s], b[s], c, 0, 0, 0);
    return c;
  }
  static __device__ __forceinline__ frag load(const float* p) {
    // two 16-byte reads: fragment addresses are only 16-byte aligned
    const f32x4 lo = *reinterpret_cast<const f32x4*>(p);
    const f32x4 hi = *reinterpret_cast<const f32x4*>(p + 4);
    frag f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[i] = lo[i];
      f[i + 4] = hi[i];
    }
    return f;
  }
  static __device__ __forceinline__ frag pack(const float* v) {
    frag f;
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = v[i];
    return f;
  }
};

__device__ __forceinline__ int acc_row(int r, int lane) { return (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3); }

}  // namespace pf
