// Forward of a hidden layer for the prediction workload (paper section 4.3:
// a pretrained model is run over the dataset and its error recorded), bf16
// operands: for every variant v,
//   O_v[r][n] = bf16(relu(sum_k A_v[r][k] W_v[k][n] + b_v[n]))
// with W_v rounded to bf16 from the fp32 master.  Per variant this is a plain
// GEMM; the input rows are shared by all variants for the first layer.
//
// One workgroup (8 waves) computes a 256-row x BN-column tile of one variant.
// The contraction runs over 32-wide column blocks, double-buffered in LDS:
// the input block (256 rows x 32) is copied as is, the weight block
// (BN units x 32 inputs, contiguous in the k-blocked master) is rounded from
// fp32 on the way in.  Waves form a 4 x 2 grid of 64 x BN/2 sub-tiles of
// 32x32x16 MFMAs.  Workgroups that share a weight tile (same variant and
// column tile, all row tiles) get consecutive dispatch slots on one XCD
// (workgroup i runs on XCD i mod 8), so the tile is fetched into that XCD's
// L2 once.
#include "gevo_internal.h"
#include "gevo_device.h"

#include <hip/hip_ext.h>

#include <type_traits>

namespace gevo {

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));   // register forms of uint4 and float4
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kGM = 256;                 // rows per tile
constexpr int kGS = 32 + 8;              // LDS row stride (bf16 elements) of both operand blocks

template <int BN>
struct GemmLds {
  static constexpr size_t a_bytes = (size_t)kGM * kGS * 2;
  static constexpr size_t b_bytes = (size_t)BN * kGS * 2;
  static constexpr size_t stage = a_bytes + b_bytes;
  static constexpr size_t bytes = 2 * stage;
};

}  // namespace

template <int BN>
__global__ __launch_bounds__(512, 1) void k_fwd_gemm(FwdGemmArgs a) {
  using O = Op<uint16_t>;
  typedef GemmLds<BN> Ly;
  constexpr int WN = BN / 2;             // columns per wave
  constexpr int TJ = WN / 32;            // 32-wide column tiles per wave
  constexpr int BU = BN / 64;            // 16-byte fp32 weight chunks per thread per block
  extern __shared__ __align__(16) char smem[];

  // dispatch slot -> (variant, column tile, row tile): slot i runs on XCD i % 8;
  // pair p = (variant, column tile) is served by XCD p % 8, its row tiles in a row
  const int nr = a.R / kGM, nn = a.Np / BN;
  const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int p = (j / nr) * 8 + xcd, rt = j % nr;
  if (p >= a.P * nn) return;
  const int v = p / nn, n0 = (p % nn) * BN, r0 = rt * kGM;
  const uint64_t vt0 = vt_now();

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, lh = lane >> 5;
  const int wm = wave & 3, wn = wave >> 2;          // 64-row band, BN/2-column half
  const int Kp = a.Kp, Np = a.Np, nkb = Kp / 32;
  const uint16_t* A = a.A + a.a_vs * v;
  const float* W = a.Wm + (size_t)v * Kp * Np;

  // two sets of staging registers (blocks kb+1 and kb+2 in flight): per set two
  // 16-byte input chunks and BU fp32 weight chunks
  u32x4_t ar[2][2];
  f32x4_t wr[2][BU];
  auto load = [&](auto setc, int kb) {
    constexpr int set = decltype(setc)::value;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = tid + 512 * u, row = c >> 2, q = c & 3;
      const int gr = r0 + row < a.R ? r0 + row : a.R - 1;        // rows past R: in-bounds re-read, never stored
      ar[set][u] = *reinterpret_cast<const u32x4_t*>(A + (size_t)gr * Kp + kb * 32 + q * 8);
    }
    const float* wb = W + ((size_t)kb * Np + n0) * 32;           // BN units x 32 inputs, contiguous
#pragma unroll
    for (int u = 0; u < BU; ++u) wr[set][u] = *reinterpret_cast<const f32x4_t*>(wb + (size_t)(tid + 512 * u) * 4);
  };
  auto store = [&](auto setc) {              // register set s goes to LDS buffer s
    constexpr int set = decltype(setc)::value, buf = set;
    uint16_t* as = reinterpret_cast<uint16_t*>(smem + buf * Ly::stage);
    uint16_t* bs = reinterpret_cast<uint16_t*>(smem + buf * Ly::stage + Ly::a_bytes);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = tid + 512 * u, row = c >> 2, q = c & 3;
      *reinterpret_cast<u32x4_t*>(as + row * kGS + q * 8) = ar[set][u];
    }
#pragma unroll
    for (int u = 0; u < BU; ++u) {
      const int c = tid + 512 * u, n = c >> 3, kq = (c & 7) * 4;
      const float f[4] = {wr[set][u][0], wr[set][u][1], wr[set][u][2], wr[set][u][3]};
      uint32_t pk[2];
      to_bf16x2(f, pk);
      *reinterpret_cast<uint2*>(bs + n * kGS + kq) = make_uint2(pk[0], pk[1]);
    }
  };

  f32x16_t acc[2][TJ];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int t = 0; t < TJ; ++t) acc[i][t] = zero16();

  // block kb: compute from LDS buffer kb&1 while the loads of block kb+2 fly
  // into register set kb&1, then store block kb+1 (set (kb+1)&1) to the other
  // buffer; the loop is unrolled by two so the register sets are static
  const std::integral_constant<int, 0> s0{};
  const std::integral_constant<int, 1> s1{};
  auto step = [&](auto setc, auto otherc, int kb) {
    constexpr int set = decltype(setc)::value;
    if (kb + 2 < nkb) load(setc, kb + 2);
    const uint16_t* as = reinterpret_cast<const uint16_t*>(smem + set * Ly::stage);
    const uint16_t* bs = reinterpret_cast<const uint16_t*>(smem + set * Ly::stage + Ly::a_bytes);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint4 af[2], bf[TJ];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = O::load(as + (wm * 64 + i * 32 + l32) * kGS + h * 16 + 8 * lh);
#pragma unroll
      for (int t = 0; t < TJ; ++t) bf[t] = O::load(bs + (wn * WN + t * 32 + l32) * kGS + h * 16 + 8 * lh);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int t = 0; t < TJ; ++t) acc[i][t] = O::mma(af[i], bf[t], acc[i][t]);
    }
    if (kb + 1 < nkb) store(otherc);
    __syncthreads();
  };
  load(s0, 0);
  if (nkb > 1) load(s1, 1);
  store(s0);
  __syncthreads();
  int kb = 0;
  for (; kb + 1 < nkb; kb += 2) {
    step(s0, s1, kb);
    step(s1, s0, kb + 1);
  }
  if (kb < nkb) step(s0, s1, kb);

  // epilogue: bias, ReLU, bf16; lane holds column l32 and rows crow(r) of each tile
  uint16_t* Out = a.O + a.o_vs * v;
#pragma unroll
  for (int t = 0; t < TJ; ++t) {
    const int n = n0 + wn * WN + t * 32 + l32;
    const float bn = a.bias[(size_t)v * Np + n];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      float f[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float z = acc[i][t][r] + bn;
        f[r] = z > 0.0f ? z : 0.0f;
      }
      uint32_t pk[8];
      to_bf16x2(f, pk);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = r0 + wm * 64 + i * 32 + crow(r, lane);
        if (row < a.R) Out[(size_t)row * Np + n] = (uint16_t)(pk[r >> 1] >> (16 * (r & 1)));
      }
    }
  }
  vt_add(a.vtime, v, vt0);
}

size_t fwd_gemm_lds_bytes(int bn) { return bn == 256 ? GemmLds<256>::bytes : GemmLds<128>::bytes; }

template <int BN>
static hipError_t launch_g(const FwdGemmArgs& a, hipStream_t s, const LaunchEv& ev) {
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_fwd_gemm<BN>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)GemmLds<BN>::bytes);
    attr = true;
  }
  const int64_t pairs = (int64_t)a.P * (a.Np / BN);
  const int64_t slots = (pairs + 7) / 8 * 8 * (a.R / kGM);
  hipExtLaunchKernelGGL((k_fwd_gemm<BN>), dim3((unsigned)slots), dim3(512), GemmLds<BN>::bytes, s, ev.start,
                        ev.stop, 0, a);
  return hipGetLastError();
}

bool fwd_gemm_supported(int Kp, int Np, int R) {
  return Kp % 32 == 0 && Kp > 0 && Np % 128 == 0 && R % kGM == 0 && R > 0;
}

hipError_t launch_fwd_gemm(const FwdGemmArgs& a, hipStream_t s, const LaunchEv& ev) {
  if (!fwd_gemm_supported(a.Kp, a.Np, a.R)) return hipErrorInvalidValue;
  return a.Np % 256 == 0 ? launch_g<256>(a, s, ev) : launch_g<128>(a, s, ev);
}

}  // namespace gevo
