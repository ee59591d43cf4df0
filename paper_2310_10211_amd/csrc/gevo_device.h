// Device-side helpers shared by the HIP kernels of libgevo (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gevo {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int crow(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// round-to-nearest-even binary32 -> bfloat16; NaN stays a quiet NaN
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// p[i] = bf16(f[2i]) | bf16(f[2i+1]) << 16 with gfx950's packed conversion
// (v_cvt_pk_bf16_f32), which rounds to nearest even and keeps NaN a quiet NaN
// exactly as f32_to_bf16_bits does, denormal inputs included, under the
// kernels' IEEE denormal mode.  gevo_check_bf16_rounding compares the two over
// every binary32 encoding.
__device__ __forceinline__ uint32_t bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t x = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2_t));
}

template <int N>
__device__ __forceinline__ void to_bf16x2(const float (&f)[N], uint32_t (&p)[N / 2]) {
#pragma unroll
  for (int i = 0; i < N / 2; ++i) p[i] = bf16x2(f[2 * i], f[2 * i + 1]);
}

template <typename S> struct Op;

template <> struct Op<uint16_t> {           // bfloat16 operands
  static constexpr int KM = 16;              // contraction per MFMA
  static constexpr int KE = 8;               // consecutive elements per lane
  static constexpr int PAD = 8;              // LDS row padding (elements)
  typedef uint4 Frag;
  __device__ __forceinline__ static Frag load(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ static Frag gather(const uint16_t* p, int stride) {
    uint4 f;
    f.x = (uint32_t)p[0] | ((uint32_t)p[stride] << 16);
    f.y = (uint32_t)p[2 * stride] | ((uint32_t)p[3 * stride] << 16);
    f.z = (uint32_t)p[4 * stride] | ((uint32_t)p[5 * stride] << 16);
    f.w = (uint32_t)p[6 * stride] | ((uint32_t)p[7 * stride] << 16);
    return f;
  }
  __device__ __forceinline__ static f32x16_t mma(Frag a, Frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  }
  __device__ __forceinline__ static uint16_t from_f32(float f) { return f32_to_bf16_bits(f); }
  __device__ __forceinline__ static float to_f32(uint16_t h) { return bf16_bits_to_f32(h); }
};

template <> struct Op<float> {              // fp32 operands
  static constexpr int KM = 2;
  static constexpr int KE = 1;
  static constexpr int PAD = 1;
  typedef float Frag;
  __device__ __forceinline__ static Frag load(const float* p) { return *p; }
  __device__ __forceinline__ static Frag gather(const float* p, int) { return *p; }
  __device__ __forceinline__ static f32x16_t mma(Frag a, Frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ __forceinline__ static float from_f32(float f) { return f; }
  __device__ __forceinline__ static float to_f32(float h) { return h; }
};

// Per-variant device time (section 4.3 scores each individual by its run
// time; here variants share launches): every wave of a kernel that works on
// one variant adds the ticks of the constant-rate device clock from its start
// to its end to that variant's counter (lane 0, one vector atomic per wave;
// a null counter array records nothing).
__device__ __forceinline__ uint64_t vt_now() { return (uint64_t)wall_clock64(); }
__device__ __forceinline__ void vt_add(unsigned long long* acc, int v, uint64_t t0) {
  if (acc && (threadIdx.x & 63) == 0) atomicAdd(acc + v, (unsigned long long)(vt_now() - t0));
}

// An opaque copy of a value: lane-dependent indices recomputed from it cannot
// be hoisted out of a loop, where dozens of them would stay live in registers
// (and be spilled) for the whole loop.
__device__ __forceinline__ int opaque(int x) {
  int y;
  asm volatile("v_mov_b32 %0, %1" : "=v"(y) : "v"(x));
  return y;
}

// LDS byte address of a pointer into shared memory.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// One direct-to-LDS load (gfx950 global_load_lds_dwordx4): lane l's 16 bytes
// at sbase + voff land at LDS address lds + 16 l.  It is an explicit
// instruction the compiler does not track; the caller waits for it with
// wait_vm and a barrier before any wave reads the bytes.  m0 is set here; no
// compiler-generated code of the kernels that use this reads m0.
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1"
      :
      : "v"(voff), "s"(sbase), "s"(lds)
      : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

__device__ __forceinline__ f32x16_t zero16() {
  f32x16_t z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

// ------------------------------------------------------------------ Philox
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64-bit products; high halves are xored with the other counter words
// and the round key, which is bumped by the Weyl constants between rounds.
__device__ __forceinline__ uint4 philox(uint4 c, uint2 k) {
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
    c = make_uint4(hi1 ^ c.y ^ k.x, lo1, hi0 ^ c.w ^ k.y, lo0);
    k.x += 0x9E3779B9u;
    k.y += 0xBB67AE85u;
  }
  return c;
}
__device__ __forceinline__ uint32_t pick(uint4 r, uint32_t i) {
  return i == 0 ? r.x : (i == 1 ? r.y : (i == 2 ? r.z : r.w));
}

}  // namespace gevo
