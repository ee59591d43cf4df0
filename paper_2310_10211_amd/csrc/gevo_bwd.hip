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
// layer l that reach LDS by direct-to-LDS loads two blocks ahead of the
// multiply, into a ring of three stages (rows of 64 bytes, 16-byte chunk c
// of row r stored at c ^ ((r >> 1) & 3), so fragment reads do not collide
// in the banks); wave w computes the 64 x BP/2 sub-tile (k half w&1, batch
// half w>>1) with 32x32x16 MFMAs, accumulating the blocks in increasing
// order.  The k tiles of one variant share an XCD (workgroup i runs on XCD
// i % 8), so the variant's gradient rows are fetched into that XCD's L2
// once.  The epilogue applies ReLU' from the activations and writes the
// gradient in columns [k][b] (and, when the layer below has a backward of
// its own, in rows [b][k]).
#include "gevo_internal.h"
#include "gevo_device.h"

#include <hip/hip_ext.h>

namespace gevo {

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kBK = 128;                 // inputs k per workgroup
constexpr int kStages = 3;               // operand ring depth (loads run two blocks ahead)

__device__ __forceinline__ f32x16_t mma32(u32x4_t a, u32x4_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}

template <int BP>
struct BwdLds {
  static constexpr int a_bytes = kBK * 64;    // W^T block [128 k][32 n] bf16
  static constexpr int b_bytes = BP * 64;     // G block [BP b][32 n]
  static constexpr int stage = a_bytes + b_bytes;
  static constexpr size_t bytes = (size_t)kStages * stage;
};

}  // namespace

template <int BP>
__global__ __launch_bounds__(256, 2) void k_bwd_gemm(BwdArgs<uint16_t> a) {
  typedef BwdLds<BP> Ly;
  constexpr int BTW = BP / 64;            // 32-wide batch tiles per wave
  constexpr int JA = kBK / 64;            // direct-to-LDS loads per wave per block: W^T rows
  constexpr int JB = BP / 64;             // and G rows (16 rows of 64 bytes per load)
  extern __shared__ __align__(16) char lds[];

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

  // Wave w loads rows 16j .. 16j+15 of each operand block for its j: load j,
  // lane l -> LDS chunk 64 j + l = row 16 j + l / 4, stored chunk l % 4,
  // which holds n chunk (l % 4) ^ ((row >> 1) & 3).
  const uint32_t lds0 = lds_addr(lds);
  const int wu = __builtin_amdgcn_readfirstlane(wave);
  uint32_t offa[JA], offb[JB];
#pragma unroll
  for (int q = 0; q < JA; ++q) {
    const int row = 16 * (JA * wave + q) + (lane >> 2);
    offa[q] = (uint32_t)row * (uint32_t)Np * 2u + (uint32_t)(((lane & 3) ^ ((row >> 1) & 3)) * 16);
  }
#pragma unroll
  for (int q = 0; q < JB; ++q) {
    const int row = 16 * (JB * wave + q) + (lane >> 2);
    offb[q] = (uint32_t)row * (uint32_t)Np * 2u + (uint32_t)(((lane & 3) ^ ((row >> 1) & 3)) * 16);
  }
  // load j of block nb (j < JA: W^T rows, else G rows) into stage nb % 3
  auto issue1 = [&](int nb, int j) {
    const uint32_t st = lds0 + (uint32_t)((nb % kStages) * Ly::stage);
    if (j < JA) dma16(wt, offa[j] + (uint32_t)nb * 64u, st + (uint32_t)((JA * wu + j) * 1024));
    else dma16(gr, offb[j - JA] + (uint32_t)nb * 64u, st + (uint32_t)(Ly::a_bytes + (JB * wu + j - JA) * 1024));
  };
  auto issue = [&](int nb) {                          // block nb into stage nb % 3: JA + JB loads
#pragma unroll
    for (int j = 0; j < JA + JB; ++j) issue1(nb, j);
  };

  const int kw = (wave & 1) * 64, bw = (wave >> 1) * (BP / 2);   // this wave's sub-tile
  f32x16_t acc[2][BTW];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jt = 0; jt < BTW; ++jt) acc[i][jt] = zero16();

  // fragment rows kw + 32i + l32 (W^T) and bw + 32jt + l32 (G) all have
  // (row >> 1) & 3 == (l32 >> 1) & 3
  const int swz = (l32 >> 1) & 3;
  issue(0);
  if (nnb > 1) {
    issue(1);
    wait_vm<JA + JB>();
  } else {
    wait_vm<0>();
  }
  __syncthreads();
  for (int nb = 0; nb < nnb; ++nb) {
    // Block nb + 2 goes into the stage of block nb - 1 (free: every wave is
    // past the barrier), one load after every second MFMA rather than all
    // at once, where the wave would wait at issue for the load path.
    const bool ld = nb + 2 < nnb;
    const char* sA = lds + (nb % kStages) * Ly::stage + (size_t)(kw + l32) * 64;
    const char* sB = lds + (nb % kStages) * Ly::stage + Ly::a_bytes + (size_t)(bw + l32) * 64;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int co = 16 * ((2 * s + lh) ^ swz);
      u32x4_t fa[2], fb[BTW];
#pragma unroll
      for (int i = 0; i < 2; ++i) fa[i] = *reinterpret_cast<const u32x4_t*>(sA + 32 * i * 64 + co);
#pragma unroll
      for (int jt = 0; jt < BTW; ++jt) fb[jt] = *reinterpret_cast<const u32x4_t*>(sB + 32 * jt * 64 + co);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jt = 0; jt < BTW; ++jt) {
          acc[i][jt] = mma32(fa[i], fb[jt], acc[i][jt]);
          constexpr int kPer = 2 * BTW;                  // MFMAs per contraction step
          const int m = s * kPer + i * BTW + jt;         // a constant after unrolling
          if ((m & 1) && (m >> 1) < JA + JB) {
            __builtin_amdgcn_sched_barrier(0);
            if (ld) issue1(nb + 2, m >> 1);
            __builtin_amdgcn_sched_barrier(0);
          }
        }
    }
    if (nb + 1 < nnb) {
      // block nb + 1 has landed (block nb + 2 may not)
      if (nb + 2 < nnb) wait_vm<JA + JB>();
      else wait_vm<0>();
      __syncthreads();
    }
  }

  // epilogue: lane l32 holds batch row bw + 32jt + l32, inputs k0 + kw +
  // 32i + crow(r).  The tile goes to LDS as bf16 rows [k][b] (stride BP + 8),
  // then every thread takes 16-byte chunks of rows: ReLU' from the
  // activations' columns [k][b] read 16 bytes at a time, and the gradient
  // columns written 16 bytes at a time.  bf16 rounding commutes with the
  // mask (bf16(0) = 0).
  constexpr int ST = BP + 8;                             // staging row stride (elements)
  static_assert((size_t)kBK * ST * 2 <= BwdLds<BP>::bytes, "staging fits the operand ring");
  const uint16_t* acv = a.Acols + a.ac_vs * v;
  uint16_t* gc = a.Gcols + a.gc_vs * v;
  uint16_t* go = a.Grows_out ? a.Grows_out + a.go_vs * v : nullptr;
  uint16_t* stg = reinterpret_cast<uint16_t*>(lds);
  __syncthreads();                                       // every wave is done with the operand ring
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jt = 0; jt < BTW; ++jt) {
      const int b = bw + 32 * jt + l32;
      uint32_t pk[8];
      {
        float f[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) f[r] = acc[i][jt][r];
        to_bf16x2(f, pk);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) stg[(kw + 32 * i + crow(r, lane)) * ST + b] = (uint16_t)(pk[r >> 1] >> (16 * (r & 1)));
      if (go) {
        // rows [b][k] keep the mask from the columns, two bytes per element
        uint32_t mk[8];
        {
          float f[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int k = k0 + kw + 32 * i + crow(r, lane);
            f[r] = bf16_bits_to_f32(acv[(size_t)k * BP + b]) > 0.0f ? acc[i][jt][r] : 0.0f;
          }
          to_bf16x2(f, mk);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)                      // inputs 8q + 4lh + 0..3 are consecutive
          *reinterpret_cast<u32x2_t*>(go + (size_t)b * Kp + k0 + kw + 32 * i + 8 * q + 4 * lh) =
              u32x2_t{mk[2 * q], mk[2 * q + 1]};
      }
    }
  __syncthreads();
  constexpr int CPR = BP / 8;                            // 16-byte chunks per row
  constexpr int NCH = kBK * CPR / 256;                   // chunks per thread
  u32x4_t am[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int ci = tid + 256 * c, row = ci / CPR, b8 = (ci % CPR) * 8;
    am[c] = *reinterpret_cast<const u32x4_t*>(acv + (size_t)(k0 + row) * BP + b8);
  }
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int ci = tid + 256 * c, row = ci / CPR, b8 = (ci % CPR) * 8;
    u32x4_t gv = *reinterpret_cast<const u32x4_t*>(stg + row * ST + b8);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t m = am[c][w];
      uint32_t keep = 0;
      if (bf16_bits_to_f32((uint16_t)(m & 0xffffu)) > 0.0f) keep |= 0xffffu;
      if (bf16_bits_to_f32((uint16_t)(m >> 16)) > 0.0f) keep |= 0xffff0000u;
      gv[w] &= keep;
    }
    *reinterpret_cast<u32x4_t*>(gc + (size_t)(k0 + row) * BP + b8) = gv;
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
