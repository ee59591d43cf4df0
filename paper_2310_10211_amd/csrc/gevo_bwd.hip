// Backward GEMM of a hidden layer with a hidden layer below, bf16 operands
// (section 6.2: the gradient of the mean loss reaches every weight through
// the chain rule): for every variant v,
//   G_{l-1}[b][k] = bf16( [A_{l-1}[b][k] > 0] * sum_n W_l[k][n] G_l[b][n] )
// with W_l the pre-update operand copy (transposed, [k][n]) and G_l the
// gradient at layer l's output in rows [b][n].  Per variant this is a plain
// GEMM with a ReLU' epilogue.
//
// One workgroup (4 waves) computes 128 inputs k x all batch rows of one
// variant, so every operand byte is read from global memory by one
// workgroup of each k tile.  The contraction runs over 32-unit blocks of
// layer l, double-buffered in LDS; wave w computes the 64 x BP/2 sub-tile
// (k half w&1, batch half w>>1) with 32x32x16 MFMAs, accumulating the blocks
// in increasing order.  The k tiles of one variant share an XCD (workgroup i
// runs on XCD i % 8), so the variant's gradient rows are fetched into that
// XCD's L2 once.  The epilogue applies ReLU' from the activations and writes
// the gradient in columns [k][b] (and, when the layer below has a backward
// of its own, in rows [b][k]).
#include "gevo_internal.h"
#include "gevo_device.h"

#include <hip/hip_ext.h>

namespace gevo {

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kBK = 128;                 // inputs k per workgroup
constexpr int kBS = 32 + 8;              // LDS row stride (bf16 elements) of both operand blocks

__device__ __forceinline__ f32x16_t mma32(u32x4_t a, u32x4_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}

template <int BP>
struct BwdLds {
  static constexpr int a_elems = kBK * kBS;   // W^T block [128 k][32 n]
  static constexpr int b_elems = BP * kBS;    // G block [BP b][32 n]
  static constexpr int stage = a_elems + b_elems;
  static constexpr size_t bytes = (size_t)2 * stage * 2;
};

}  // namespace

template <int BP>
__global__ __launch_bounds__(256, 2) void k_bwd_gemm(BwdArgs<uint16_t> a) {
  typedef BwdLds<BP> Ly;
  constexpr int BTW = BP / 64;            // 32-wide batch tiles per wave
  constexpr int UA = kBK * 4 / 256;       // 16-byte chunks per thread of the W^T block
  constexpr int UB = BP * 4 / 256;        // and of the G block
  extern __shared__ __align__(16) uint16_t lds[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, lh = lane >> 5;
  int v, kt;
  {
    const int gx = gridDim.x, total = gx * gridDim.y, i = blockIdx.y * gx + blockIdx.x;
    const int j = total % 8 == 0 ? (i % 8) * (total / 8) + i / 8 : i;
    v = j / gx;
    kt = j % gx;
  }
  const uint64_t vt0 = vt_now();
  const int Kp = a.Kp, Np = a.Np, nnb = Np / 32;
  const int k0 = kt * kBK;
  const uint16_t* wt = a.Wt + (size_t)v * Kp * Np + (size_t)k0 * Np;   // rows k0.., [k][n]
  const uint16_t* gr = a.Grows + a.gr_vs * v;                           // [b][n]

  u32x4_t sa[UA], sb[UB];
  auto load = [&](int nb) {
#pragma unroll
    for (int q = 0; q < UA; ++q) {
      const int i = tid + 256 * q;
      sa[q] = *reinterpret_cast<const u32x4_t*>(wt + (size_t)(i >> 2) * Np + nb * 32 + (i & 3) * 8);
    }
#pragma unroll
    for (int q = 0; q < UB; ++q) {
      const int i = tid + 256 * q;
      sb[q] = *reinterpret_cast<const u32x4_t*>(gr + (size_t)(i >> 2) * Np + nb * 32 + (i & 3) * 8);
    }
  };
  auto store = [&](int buf) {
    uint16_t* sA = lds + buf * Ly::stage;
    uint16_t* sB = sA + Ly::a_elems;
#pragma unroll
    for (int q = 0; q < UA; ++q) {
      const int i = tid + 256 * q;
      *reinterpret_cast<u32x4_t*>(sA + (i >> 2) * kBS + (i & 3) * 8) = sa[q];
    }
#pragma unroll
    for (int q = 0; q < UB; ++q) {
      const int i = tid + 256 * q;
      *reinterpret_cast<u32x4_t*>(sB + (i >> 2) * kBS + (i & 3) * 8) = sb[q];
    }
  };

  const int kw = (wave & 1) * 64, bw = (wave >> 1) * (BP / 2);   // this wave's sub-tile
  f32x16_t acc[2][BTW];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jt = 0; jt < BTW; ++jt) acc[i][jt] = zero16();

  load(0);
  store(0);
  __syncthreads();
  for (int nb = 0; nb < nnb; ++nb) {
    const int buf = nb & 1;
    if (nb + 1 < nnb) load(nb + 1);
    const uint16_t* sA = lds + buf * Ly::stage + (kw + l32) * kBS + 8 * lh;
    const uint16_t* sB = lds + buf * Ly::stage + Ly::a_elems + (bw + l32) * kBS + 8 * lh;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      u32x4_t fa[2], fb[BTW];
#pragma unroll
      for (int i = 0; i < 2; ++i) fa[i] = *reinterpret_cast<const u32x4_t*>(sA + 32 * i * kBS + 16 * s);
#pragma unroll
      for (int jt = 0; jt < BTW; ++jt) fb[jt] = *reinterpret_cast<const u32x4_t*>(sB + 32 * jt * kBS + 16 * s);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jt = 0; jt < BTW; ++jt) acc[i][jt] = mma32(fa[i], fb[jt], acc[i][jt]);
    }
    if (nb + 1 < nnb) store(buf ^ 1);                    // its old block was last read before the previous barrier
    __syncthreads();
  }

  // epilogue: lane l32 holds batch row bw + 32jt + l32, inputs k0 + kw + 32i + crow(r)
  const uint16_t* acv = a.Acols + a.ac_vs * v;
  uint16_t* gc = a.Gcols + a.gc_vs * v;
  uint16_t* go = a.Grows_out ? a.Grows_out + a.go_vs * v : nullptr;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jt = 0; jt < BTW; ++jt) {
      const int b = bw + 32 * jt + l32;
      float f[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int k = k0 + kw + 32 * i + crow(r, lane);
        const float av = bf16_bits_to_f32(acv[(size_t)k * BP + b]);
        f[r] = av > 0.0f ? acc[i][jt][r] : 0.0f;
      }
      uint32_t pk[8];
      to_bf16x2(f, pk);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int k = k0 + kw + 32 * i + crow(r, lane);
        gc[(size_t)k * BP + b] = (uint16_t)(pk[r >> 1] >> (16 * (r & 1)));
      }
      if (go)
#pragma unroll
        for (int q = 0; q < 4; ++q)                      // inputs 8q + 4lh + 0..3 are consecutive
          *reinterpret_cast<u32x2_t*>(go + (size_t)b * Kp + k0 + kw + 32 * i + 8 * q + 4 * lh) =
              u32x2_t{pk[2 * q], pk[2 * q + 1]};
    }
  vt_add(a.vtime, v, vt0);
}

bool bwd_gemm_supported(int Kp, int Np, int Bp) {
  return Kp % kBK == 0 && Kp > 0 && Np % 32 == 0 && Np > 0 && (Bp == 128 || Bp == 256);
}

template <int BP>
static hipError_t launch_b(const BwdArgs<uint16_t>& a, int P, hipStream_t s, const LaunchEv& ev) {
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_bwd_gemm<BP>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)BwdLds<BP>::bytes);
    attr = true;
  }
  hipExtLaunchKernelGGL((k_bwd_gemm<BP>), dim3(a.Kp / kBK, P), dim3(256), BwdLds<BP>::bytes, s, ev.start, ev.stop, 0,
                        a);
  return hipGetLastError();
}

hipError_t launch_bwd_gemm(const BwdArgs<uint16_t>& a, int P, hipStream_t s, const LaunchEv& ev) {
  if (!bwd_gemm_supported(a.Kp, a.Np, a.Bp)) return hipErrorInvalidValue;
  return a.Bp == 256 ? launch_b<256>(a, P, s, ev) : launch_b<128>(a, P, s, ev);
}

}  // namespace gevo
