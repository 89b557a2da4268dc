// Device-side building blocks shared by the gfx950 kernels of the denoise loop.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "vla_internal.h"

typedef uint16_t bf16_t;  // bf16 storage
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

#define VLA_DEV __device__ __forceinline__

VLA_DEV float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// float -> bf16, round to nearest even (hardware conversion on gfx950).
VLA_DEV bf16_t f2bf(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(bf16_t, h);
}

VLA_DEV uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

// Elements per 16-byte vector and conversion helpers, per storage type.
template <typename T> struct ElemTraits;
template <> struct ElemTraits<float> {
  static constexpr int E = 4;
  static VLA_DEV float to_f(float v) { return v; }
  static VLA_DEV float from_f(float v) { return v; }
};
template <> struct ElemTraits<bf16_t> {
  static constexpr int E = 8;
  static VLA_DEV float to_f(bf16_t v) { return bf2f(v); }
  static VLA_DEV bf16_t from_f(float v) { return f2bf(v); }
};

// Pack 16 bytes worth of float values (E of them) into the storage type.
VLA_DEV uint4 pack16(const float* v, float) {
  return make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                    __float_as_uint(v[3]));
}
VLA_DEV uint4 pack16(const float* v, bf16_t) {
  return make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                    pack_bf16x2(v[6], v[7]));
}
VLA_DEV void unpack16(uint4 u, float* v, float) {
  v[0] = __uint_as_float(u.x); v[1] = __uint_as_float(u.y);
  v[2] = __uint_as_float(u.z); v[3] = __uint_as_float(u.w);
}
VLA_DEV void unpack16(uint4 u, float* v, bf16_t) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

// One 16-byte A fragment times one 16-byte B fragment into a 16x16 fp32 tile.
// bf16: one v_mfma_f32_16x16x32_bf16 (8 k-values per lane).
// fp32: four v_mfma_f32_16x16x4_f32 (one k-value per lane each).
VLA_DEV void mma16(f32x4& acc, uint4 a, uint4 b, bf16_t) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
VLA_DEV void mma16(f32x4& acc, uint4 a, uint4 b, float) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// 16-byte load from global memory.  The explicit global address space (on a
// native vector type: uint4's copy constructor would take a generic
// reference) keeps the compiler from emitting a flat load where it cannot
// prove the pointer global, e.g. one read from memory.  Flat loads also count
// on lgkmcnt, so every wait for an LDS read would wait for them too.
typedef unsigned gv4u_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const gv4u_t global_v4u;
VLA_DEV uint4 ldg16(const void* p) {
  const gv4u_t v = *(const global_v4u*)(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}
VLA_DEV void stg16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }

// Activations (fp32).  GELU uses the tanh form.  Both use the hardware
// reciprocal (about 1 ulp) instead of a correctly rounded division; the
// results feed bf16 operands.  tanh(y) = 1 - 2 / (1 + e^(2y)): for large |y|
// the exponential saturates to inf or 0 and the result to +-1.
VLA_DEV float silu_f(float x) { return x * __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }
VLA_DEV float tanh_f(float y) { return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + __expf(2.0f * y)); }
VLA_DEV float gelu_tanh_f(float x) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float inner = k0 * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.0f + tanh_f(inner));
}
VLA_DEV float act_f(int act, float x) {
  switch (act) {
    case ACT_SILU: return silu_f(x);
    case ACT_GELU: return gelu_tanh_f(x);
    case ACT_RELU2: { float r = fmaxf(x, 0.0f); return r * r; }
    default: return x;
  }
}

// Sum over the 16 lanes that share lane/16 (the columns of one MFMA tile row group).
VLA_DEV float sum16(float v) {
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 8, 64);
  return v;
}
VLA_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
VLA_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Split-K arrival: every thread has stored its partials; returns true in all
// threads of the last workgroup to arrive on `counter` (which it resets).
VLA_DEV bool splitk_arrive_last(unsigned* counter, unsigned nsplit, int* lds_flag) {
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned old = atomicAdd(counter, 1u);
    bool last = (old == nsplit - 1);
    if (last) atomicExch(counter, 0u);
    *lds_flag = last ? 1 : 0;
  }
  __syncthreads();
  bool last = *lds_flag != 0;
  if (last) __threadfence();
  return last;
}

// ---- direct-to-LDS staging (the tiled GEMMs) ---------------------------------
typedef unsigned v4u __attribute__((ext_vector_type(4)));  // one 16-byte LDS slot

// One wave-wide global_load_lds_dwordx4: lane l's 16 bytes at g land in LDS
// at wave-uniform lds + 16 l.  Written as asm so that the compiler adds no
// waits of its own for it; the kernel's explicit vmcnt waits and barriers
// order it against the LDS reads.
VLA_DEV void dma16(const void* g, v4u* lds) {
  typedef __attribute__((address_space(3))) v4u lds_v4u;
  const unsigned off = (unsigned)(uintptr_t)(lds_v4u*)lds;  // byte offset in the workgroup's LDS
  const unsigned base = __builtin_amdgcn_readfirstlane(off);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" : : "s"(base), "v"(g) : "memory", "m0");
}

// Workgroup barrier after this wave's LDS reads have completed; the memory
// clobber keeps the compiler from moving LDS accesses across it.
VLA_DEV void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" : : : "memory"); }

VLA_DEV constexpr unsigned vm_wait(int n) {  // s_waitcnt: vmcnt(n), no wait on the other counters
  return (unsigned)((n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8));
}
