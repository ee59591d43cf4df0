// Fused per-variant training kernel for two-layer nets (bf16 operands, fp32
// master weights): one persistent workgroup owns one variant for a whole run
// of SGD steps (paper section 6.2 update rule; fitness by retraining, section
// 4.3).  Variants never exchange data, so workgroups are fully independent.
//
// Per step t, for hidden width HP and batch tile BP
// (one wave per 32 hidden units, HP/32 waves):
//   A1 = relu(Z1 + b1): rows -> LDS (logits operand), bf16 pairs kept in
//        registers (dW2 operand; a nonzero pair half is also ReLU')
//   logits^T = W2 A1^T + b2 (one batch tile per wave, so a lane holds one
//        row's classes, split over lanes l and l+32); softmax cross-entropy,
//        argmax and G2 = (p - y) fl(1/b) in the same registers; G2 -> LDS in
//        both orientations, fp32 G2 -> LDS columns for db2
//   dW2 = G2^T A1,  G1 = (G2 W2) * ReLU' (pre-update W2),  db1, db2;
//        W2 (fp32 master in LDS), b2, b1 updated
//   then, streaming the fp32 master W1 once per 32-column block k:
//     dW1[k][n] = sum_b X_t[b][k] G1[b][n]           (MFMA, contraction = batch)
//     W1 = mask ? fl(W1 - fl(lr dW1)) : +0           (float4 in place)
//     Z1'[b][n] += sum_k X_{t+1}[b][k] W1new[k][n]   (forward of step t+1)
// The accumulator layout of a 32x32 MFMA gives lane l the column l%32 and the
// rows 8(r/4) + 4(l/32) + r%4 of register r.  Taking the eight registers
// 8s..8s+7 of a tile as the operand of contraction step s (i.e. contracting
// over the rows {16s + 4(l/32) + 0..3, 16s + 8 + 4(l/32) + 0..3}) lets a tile
// produced as an accumulator feed the next MFMA directly; the other operand is
// read from LDS with the same row permutation.  This is how G1 (accumulators
// over b) feeds dW1, how A1 feeds dW2, how the lane's own W2 master values
// feed G1, and how the updated W1 (accumulators over k) feeds the forward pass
// without leaving registers.
//
// W1 is kept in a register image: in block kb, wave w's q-th 16-byte load of
// every lane reads one contiguous KiB (lane l32 + 32 lh holds inputs
// 8q + 4lh + 0..3 of unit 32w + l32), and the mask words are block-major, so
// every W1 load and store instruction covers whole cache lines.
// The W1 stream is software-pipelined one block ahead and the shared X blocks
// two blocks ahead; the block loop is unrolled by two with alternating
// register sets.  All these loads are explicit instructions with one explicit
// wait at the top of the next block, so no wait for a compiler-visible load can
// also drain the prefetch.  The X rows of a step are stored block-major
// ([Kp/32][B][32]), so one block's rows are a contiguous 8 KB, and each
// workgroup starts its passes at a different column block, so the workgroups
// sharing an L2 do not all request the same X lines at once.
#include "gevo_internal.h"
#include "gevo_device.h"

#include <hip/hip_ext.h>
#include <math.h>

#include <type_traits>

namespace gevo {

namespace {

__device__ __forceinline__ uint4 ld2x8(const uint16_t* p0, const uint16_t* p1) {
  const uint2 lo = *reinterpret_cast<const uint2*>(p0);
  const uint2 hi = *reinterpret_cast<const uint2*>(p1);
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}

__device__ __forceinline__ uint32_t pack2(uint16_t lo, uint16_t hi) { return (uint32_t)lo | ((uint32_t)hi << 16); }

__device__ __forceinline__ uint4 pack8(const uint16_t* u) {
  return make_uint4(pack2(u[0], u[1]), pack2(u[2], u[3]), pack2(u[4], u[5]), pack2(u[6], u[7]));
}

// bf16 element r of eight packed pairs
__device__ __forceinline__ uint16_t half_of(const uint32_t* p, int r) { return (uint16_t)(p[r >> 1] >> (16 * (r & 1))); }

__device__ __forceinline__ float f4get(const float4& f, int i) {
  return i == 0 ? f.x : (i == 1 ? f.y : (i == 2 ? f.z : f.w));
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));   // register-operand forms of float4
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));   // and uint4

// 16x16x32 bf16 MFMA: lane l supplies row (A) / column (B) l%16, contraction
// elements 8(l/16) .. 8(l/16)+7; the accumulator gives lane l the column l%16
// and the rows 4(l/16) .. 4(l/16)+3.
__device__ __forceinline__ f32x4_t mma16(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}

}  // namespace

template <int HP, int BP>
struct Fused2Lds {
  static constexpr int NW = HP / 32;     // waves
  static constexpr int BT = BP / 32;     // batch tiles
  static constexpr int NBS = BP / 16;    // contraction steps over the batch
  static constexpr int XR = 32 + 8;      // X row block [BP][32]
  static constexpr int XC = BP + 8;      // X col block [32][BP]
  static constexpr int AS = HP + 8;      // A1 rows [BP][HP]
  static constexpr int W2S = HP + 8;     // W2 bf16 operand [32][HP]
  static constexpr int GS = 32 + 8;      // G2 rows [BP][32]
  static constexpr int GTS = BP + 8;     // G2 columns [32][BP]
  // region X, block loop: two X row blocks and two X column blocks
  static constexpr size_t xr = 0;
  static constexpr size_t xc = xr + 2ull * BP * XR * 2;
  static constexpr size_t xend = xc + 2ull * 32 * XC * 2;
  // region X, output-layer phase
  static constexpr size_t g2 = 0;
  static constexpr int ZGS = BP + 1;     // fp32 G2 columns [32][BP]
  static constexpr size_t g2t = g2 + (size_t)BP * GS * 2;
  static constexpr size_t zg = g2t + 32ull * GTS * 2;       // [32][ZGS] fp32
  static constexpr size_t yl = zg + 32ull * ZGS * 4;        // [BP] labels of the step
  static constexpr size_t send = yl + (size_t)BP * 4;
  static_assert(send <= xend, "output-layer scratch must fit in the X buffers");
  // region A: A1 rows in the output-layer phase, G1 operand slots in the block loop
  static constexpr size_t a1 = (xend + 15) / 16 * 16;
  static constexpr size_t a1_bytes = (size_t)BP * AS * 2;
  static_assert((size_t)NW * NBS * 64 * 16 <= a1_bytes, "G1 slots must fit in the A1 region");
  // persistent: W2 bf16 operand, W2 fp32 master (swizzled rows), b2
  static constexpr size_t w2 = a1 + a1_bytes;
  static constexpr size_t w2m = (w2 + 32ull * W2S * 2 + 15) / 16 * 16;
  static constexpr size_t b2 = w2m + (size_t)HP * 32 * 4;
  static constexpr int NDP = 2 * NW;     // db2 partial sums per class
  static constexpr size_t dbp = b2 + 32 * 4;                // [NDP][32] fp32
  static constexpr size_t rce = dbp + (size_t)NDP * 32 * 4; // [BP] fp64 per-row loss
  static constexpr size_t rco = rce + (size_t)BP * 8;       // [BP] per-row hit
  static constexpr size_t bytes = rco + (size_t)BP * 4;
  static_assert(rce % 8 == 0, "fp64 row losses must be 8-byte aligned");
};

template <int HP, int BP>
__global__ __launch_bounds__(2 * HP, 1) void k_fused2(Fused2Args a) {
  using O = Op<uint16_t>;
  typedef Fused2Lds<HP, BP> Ly;
  constexpr int NW = Ly::NW;                 // waves, one per 32 hidden units
  constexpr int NT = 64 * NW;                // threads
  constexpr int XU = (4 * BP + NT - 1) / NT; // 16-byte X chunks per thread per block
  constexpr int BT = Ly::BT;
  constexpr int NBS = Ly::NBS;
  extern __shared__ __align__(16) char smem[];
  uint16_t* xr = reinterpret_cast<uint16_t*>(smem + Ly::xr);
  uint16_t* xc = reinterpret_cast<uint16_t*>(smem + Ly::xc);
  uint16_t* g2 = reinterpret_cast<uint16_t*>(smem + Ly::g2);
  uint16_t* g2t = reinterpret_cast<uint16_t*>(smem + Ly::g2t);
  float* zg = reinterpret_cast<float*>(smem + Ly::zg);
  int* yl = reinterpret_cast<int*>(smem + Ly::yl);
  float* dbp = reinterpret_cast<float*>(smem + Ly::dbp);
  double* rce = reinterpret_cast<double*>(smem + Ly::rce);
  unsigned int* rco = reinterpret_cast<unsigned int*>(smem + Ly::rco);
  uint16_t* a1 = reinterpret_cast<uint16_t*>(smem + Ly::a1);
  uint4* g1s = reinterpret_cast<uint4*>(smem + Ly::a1);
  uint16_t* w2 = reinterpret_cast<uint16_t*>(smem + Ly::w2);
  float* w2m = reinterpret_cast<float*>(smem + Ly::w2m);
  float* b2s = reinterpret_cast<float*>(smem + Ly::b2);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, lh = lane >> 5;
  const int v = blockIdx.x;
  const uint64_t vt0 = vt_now();
  const int Kp = a.Kp, nkb = Kp / 32;
  const int n = wave * 32 + l32;             // hidden unit of this lane's column
  float* W1 = a.W1 + (size_t)v * HP * Kp;
  const uint32_t* m1 = a.m1 + (size_t)v * HP * nkb;
  float* W2 = a.W2 + (size_t)v * 32 * HP;
  const uint32_t* m2 = a.m2 + (size_t)v * 32 * (HP / 32);
  const float lrv = a.lr[v];
  const float lrv2 = a.lr2 ? a.lr2[v] : lrv;   // output layer (the hidden layer's rate is 0 when removed)
  // Every pass visits the column blocks in the order rot, rot+1, ... (mod nkb).
  // All workgroups read the same shared X blocks; workgroup v runs on XCD
  // v mod 8, and staggering the start block over the workgroups of one XCD
  // keeps them from requesting the same L2 lines at the same moment.  The
  // forward's fp32 sum over blocks follows this order.
  const int rot = (v >> 3) % nkb;
  auto phys = [&](int j) { return j + rot < nkb ? j + rot : j + rot - nkb; };

  // Output layer, resident for the whole run: the fp32 master of this lane's
  // 16 (class, unit) pairs lives in LDS row n (4-float chunk j stored at chunk
  // j ^ (n & 7), which spreads the lanes of a row read over all banks); the
  // bf16 operand copy [class][unit] feeds the logits; mask bits in a register.
  float* w2row = w2m + n * 32;
  const int sw = n & 7;
  uint32_t m2bits = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float f[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * q + i, c = crow(r, lane);
      f[i] = W2[((size_t)wave * 32 + c) * 32 + l32];
      w2[c * Ly::W2S + n] = O::from_f32(f[i]);
      m2bits |= ((m2[c * (HP / 32) + wave] >> l32) & 1u) << r;
    }
    *reinterpret_cast<float4*>(w2row + (((2 * q + lh) ^ sw) << 2)) = make_float4(f[0], f[1], f[2], f[3]);
  }
  if (tid < 32) b2s[tid] = a.b2[(size_t)v * 32 + tid];
  float b1v = a.b1[(size_t)v * HP + n];
  const bool b1k = (a.bm1[(size_t)v * (HP / 32) + wave] >> l32) & 1u;   // this unit's bias is trained
  const bool b2k = tid < 32 && ((a.bm2[v] >> (tid & 31)) & 1u);          // class tid's bias is trained
  double ce_tot = 0.0;
  unsigned long long corr_tot = 0;
  const int tot_tid = (NW - 1) * 64;          // thread that keeps the loss / hit totals
  if (tid == tot_tid) {
    ce_tot = a.ce_acc[v];
    corr_tot = a.correct_acc[v];
  }

  f32x16_t zacc[BT];

  // Prefetch registers of the block loop: two sets of X staging registers
  // (block kb+1 waiting for its LDS buffer, block kb+2 in flight) and two sets
  // of W1 master registers (block kb in use, block kb+1 in flight).  Every load
  // into them is an explicit instruction with an explicit wait: a load the
  // compiler tracked into a loop-carried register would make it wait for all
  // outstanding memory operations at the loop head.
  u32x4_t xAr[XU], xAc[XU], xBr[XU], xBc[XU];
  f32x4_t wA[4], wB[4];
  uint32_t mA = 0, mB = 0;
  int ylab = -1;
  // X block of visit j (clamped: past the end an in-bounds re-read whose value
  // is never stored; threads past the block's chunks re-read its last chunk)
  auto load_x = [&](auto updc, int tu, auto fwdc, int tf, int j, int td, u32x4_t (&xrn)[XU], u32x4_t (&xcn)[XU]) {
    constexpr bool upd = decltype(updc)::value, fwd = decltype(fwdc)::value;
    const uint16_t* xrs = a.xrows + (size_t)tf * BP * Kp;
    const uint16_t* xcs = a.xcols + (size_t)tu * Kp * BP;
    const int kc = phys(j < nkb ? j : nkb - 1);
#pragma unroll
    for (int u = 0; u < XU; ++u) {
      const int i = td + NT * u < 4 * BP ? td + NT * u : 4 * BP - 1;
      if constexpr (fwd) {                         // rows block-major: block kc is BP x 32 contiguous
        const uint16_t* p = xrs + (size_t)kc * BP * 32 + (size_t)i * 8;
        asm volatile("global_load_dwordx4 %0, %1, off" : "=&v"(xrn[u]) : "v"(p) : "memory");
      }
      if constexpr (upd) {
        const uint16_t* p = xcs + (size_t)(kc * 32 + i / (BP / 8)) * BP + (i % (BP / 8)) * 8;
        asm volatile("global_load_dwordx4 %0, %1, off" : "=&v"(xcn[u]) : "v"(p) : "memory");
      }
    }
  };
  auto store_x = [&](auto updc, auto fwdc, int buf, int td, const u32x4_t (&xrn)[XU], const u32x4_t (&xcn)[XU]) {
    constexpr bool upd = decltype(updc)::value, fwd = decltype(fwdc)::value;
#pragma unroll
    for (int u = 0; u < XU; ++u) {
      const int i = td + NT * u;
      if (i < 4 * BP) {
        if constexpr (fwd) {
          const int b = i >> 2, q = i & 3;
          *reinterpret_cast<u32x4_t*>(xr + buf * BP * Ly::XR + b * Ly::XR + q * 8) = xrn[u];
        }
        if constexpr (upd) {
          const int k = i / (BP / 8), q = i % (BP / 8);
          *reinterpret_cast<u32x4_t*>(xc + buf * 32 * Ly::XC + k * Ly::XC + q * 8) = xcn[u];
        }
      }
    }
  };
  // W1 block of visit j for this wave (and its mask words when updating)
  auto load_w = [&](auto updc, int j, int td, f32x4_t (&wn)[4], uint32_t& mn) {
    constexpr bool upd = decltype(updc)::value;
    const int kb = phys(j);
    const float* wp = W1 + ((size_t)kb * NW + wave) * 1024 + (td & 63) * 4;
    if constexpr (upd) {
      const uint32_t* mp = m1 + (size_t)kb * HP + wave * 32 + (td & 31);
      asm volatile(
          "global_load_dwordx4 %0, %5, off\n\t"
          "global_load_dwordx4 %1, %5, off offset:1024\n\t"
          "global_load_dwordx4 %2, %5, off offset:2048\n\t"
          "global_load_dwordx4 %3, %5, off offset:3072\n\t"
          "global_load_dword %4, %6, off"
          : "=&v"(wn[0]), "=&v"(wn[1]), "=&v"(wn[2]), "=&v"(wn[3]), "=&v"(mn)
          : "v"(wp), "v"(mp)
          : "memory");
    } else {
      asm volatile(
          "global_load_dwordx4 %0, %4, off\n\t"
          "global_load_dwordx4 %1, %4, off offset:1024\n\t"
          "global_load_dwordx4 %2, %4, off offset:2048\n\t"
          "global_load_dwordx4 %3, %4, off offset:3072"
          : "=&v"(wn[0]), "=&v"(wn[1]), "=&v"(wn[2]), "=&v"(wn[3])
          : "v"(wp)
          : "memory");
      mn = 0u;
    }
  };
  // head of the next pass over the input columns: X blocks 0 and 1, W1 block 0
  // and its mask words (in this order), then the labels of the step whose loss
  // the pass prepares
  auto issue_head = [&](auto updc, int tu, auto fwdc, int tf, int td) {
    constexpr bool fwd = decltype(fwdc)::value;
    load_x(updc, tu, fwdc, tf, 0, td, xAr, xAc);
    load_x(updc, tu, fwdc, tf, 1, td, xBr, xBc);
    load_w(updc, 0, td, wA, mA);
    if (fwd && td < BP) ylab = a.labels[(size_t)tf * BP + td];
  };

  // visit kb of a pass (column block phys(kb)): dW1 + update (step tu) and/or
  // forward accumulation of step tf; wc/mc hold visit kb's W1 block, wn/mn
  // receive visit kb+1's, xl receives X of visit kb+2, xs holds X of visit kb+1
  // for the other buffer
  auto kblock = [&](auto firstc, auto updc, int tu, auto fwdc, int tf, int kb, int td, f32x4_t (&wc)[4],
                    uint32_t& mc, f32x4_t (&wn)[4], uint32_t& mn, u32x4_t (&xlr)[XU], u32x4_t (&xlc)[XU],
                    u32x4_t (&xsr)[XU], u32x4_t (&xsc)[XU]) {
    constexpr bool upd = decltype(updc)::value, fwd = decltype(fwdc)::value;
    const int lane = td & 63, l32 = lane & 31, lh = lane >> 5, n = wave * 32 + l32;
    const int buf = kb & 1;
    const bool more = kb + 1 < nkb;
    // Block kb's W1 words and X block kb+1 were issued one block earlier, and
    // vector memory operations retire in issue order.  After them that block
    // issued only its four W1 stores (when updating), which may stay in
    // flight; block 0 follows the head and waits for everything.
    constexpr int NS = (decltype(firstc)::value || !upd) ? 0 : 4;
    asm volatile("s_waitcnt vmcnt(%5)"
                 : "+v"(wc[0]), "+v"(wc[1]), "+v"(wc[2]), "+v"(wc[3]), "+v"(mc)
                 : "n"(NS)
                 : "memory");
#pragma unroll
    for (int u = 0; u < XU; ++u) asm volatile("" : "+v"(xsr[u]), "+v"(xsc[u]));
    load_x(updc, tu, fwdc, tf, kb + 2, td, xlr, xlc);
    load_w(updc, more ? kb + 1 : kb, td, wn, mn);   // the last block re-reads itself (in bounds, unused)
    const uint16_t* xcb = xc + buf * 32 * Ly::XC;
    const uint16_t* xrb = xr + buf * BP * Ly::XR;
    float wnew[16];
    if constexpr (upd) {
      f32x16_t dacc = zero16();
#pragma unroll
      for (int s = 0; s < NBS; ++s) {
        const uint16_t* pp = xcb + l32 * Ly::XC + 16 * s + 4 * lh;
        dacc = O::mma(ld2x8(pp, pp + 8), g1s[(wave * NBS + s) * 64 + lane], dacc);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kl = 8 * (r >> 2) + 4 * lh + (r & 3);
        const bool keep = (mc >> kl) & 1u;
        wnew[r] = keep ? __fsub_rn(wc[r >> 2][r & 3], __fmul_rn(lrv, dacc[r])) : 0.0f;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(W1 + (((size_t)phys(kb) * NW + wave) * 4 + q) * 256 + lane * 4) =
            make_float4(wnew[4 * q], wnew[4 * q + 1], wnew[4 * q + 2], wnew[4 * q + 3]);
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) wnew[r] = wc[r >> 2][r & 3];
    }
    if constexpr (fwd) {
      uint32_t pw[8];
      to_bf16x2(wnew, pw);
      const uint4 wb[2] = {make_uint4(pw[0], pw[1], pw[2], pw[3]), make_uint4(pw[4], pw[5], pw[6], pw[7])};
#pragma unroll
      for (int T = 0; T < BT; ++T)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const uint16_t* pp = xrb + (32 * T + l32) * Ly::XR + 16 * s2 + 4 * lh;
          zacc[T] = O::mma(ld2x8(pp, pp + 8), wb[s2], zacc[T]);
        }
    }
    if (more) store_x(updc, fwdc, buf ^ 1, td, xsr, xsc);
    __syncthreads();
  };

  // one pass over the input columns (head already issued): optional dW1 +
  // update (step tu), optional forward accumulation of step tf into zacc
  auto kloop = [&](auto updc, int tu, auto fwdc, int tf, int td) {
    const std::true_type first{};
    const std::false_type later{};
    if constexpr (decltype(fwdc)::value) {
#pragma unroll
      for (int T = 0; T < BT; ++T) zacc[T] = zero16();
    }
    __syncthreads();                           // the output-layer scratch shares the X buffers
    // X block 0 is the oldest operation of the head; X block 1 and W1 block 0
    // (NX + NL operations) may stay in flight
    constexpr int NX = (decltype(fwdc)::value ? XU : 0) + (decltype(updc)::value ? XU : 0);
    constexpr int NL = decltype(updc)::value ? 5 : 4;
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(NX + NL) : "memory");
#pragma unroll
    for (int u = 0; u < XU; ++u) asm volatile("" : "+v"(xAr[u]), "+v"(xAc[u]));
    store_x(updc, fwdc, 0, td, xAr, xAc);
    __syncthreads();
    // block 0, then whole pairs of blocks (alternating register sets), then an
    // odd last block: no branch inside the loop body skips a block
    kblock(first, updc, tu, fwdc, tf, 0, td, wA, mA, wB, mB, xAr, xAc, xBr, xBc);
    int kb = 1;
    for (; kb + 1 < nkb; kb += 2) {
      kblock(later, updc, tu, fwdc, tf, kb, td, wB, mB, wA, mA, xBr, xBc, xAr, xAc);
      kblock(later, updc, tu, fwdc, tf, kb + 1, td, wA, mA, wB, mB, xAr, xAc, xBr, xBc);
    }
    if (kb < nkb) kblock(later, updc, tu, fwdc, tf, kb, td, wB, mB, wA, mA, xBr, xBc, xAr, xAc);
    // the last blocks' (unused) prefetches and stores land before their registers are reused
    asm volatile("s_waitcnt vmcnt(0)"
                 : "+v"(wA[0]), "+v"(wA[1]), "+v"(wA[2]), "+v"(wA[3]), "+v"(mA), "+v"(wB[0]), "+v"(wB[1]),
                   "+v"(wB[2]), "+v"(wB[3]), "+v"(mB)
                 :
                 : "memory");
#pragma unroll
    for (int u = 0; u < XU; ++u) asm volatile("" : "+v"(xAr[u]), "+v"(xAc[u]), "+v"(xBr[u]), "+v"(xBc[u]));
  };
  const std::true_type on{};
  const std::false_type off{};

  // output layer, end of a step: b2 -= lr * sum of the db2 partials, and the
  // per-row losses and hits added to the totals (fixed order)
  auto finish_out = [&]() {
    if (tid < 32) {
      float db = 0.0f;
#pragma unroll
      for (int part = 0; part < Ly::NDP; ++part) db += dbp[part * 32 + tid];
      b2s[tid] = b2k ? __fsub_rn(b2s[tid], __fmul_rn(lrv2, db)) : 0.0f;
    }
    if (wave == NW - 1) {
      double sc = 0.0;
      unsigned int co = 0;
      for (int r = lane; r < BP; r += 64) { sc += rce[r]; co += rco[r]; }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) { sc += __shfl_xor(sc, off); co += __shfl_xor(co, off); }
      if (lane == 0) { ce_tot += sc; corr_tot += co; }
    }
  };

  // prologue: forward of the first step
  issue_head(off, 0, on, a.t0, tid);
  kloop(off, 0, on, a.t0, tid);

  for (int t = a.t0; t < a.t1; ++t) {
    // Lane-dependent indices are recomputed each step from an opaque copy of
    // the lane id: hoisted out of the loop they would occupy dozens of long-lived
    // address registers and be spilled to scratch (each reload is a memory round trip).
    int tid_step;
    asm volatile("v_mov_b32 %0, %1" : "=v"(tid_step) : "v"(tid));
    const int lane = tid_step & 63, l32 = lane & 31, lh = lane >> 5, n = wave * 32 + l32;
    float* w2row = w2m + n * 32;
    const int sw = n & 7;
    const int64_t r0 = (int64_t)t * a.B;
    const int bt = (int)((a.n - r0) < a.B ? (a.n - r0) : a.B);
    const float scale = __fdiv_rn(1.0f, (float)bt);
    // ---- the previous step's output-layer bias update and loss / hit totals
    //      (its partial sums waited in LDS during the block loop)
    if (t > a.t0) finish_out();
    // ---- A1 = relu(Z1 + b1): rows -> LDS, bf16 operand pairs in registers
    //      (a nonzero bf16 A1 value is also the ReLU' of its element)
    uint4 a1p[NBS];
#pragma unroll
    for (int T = 0; T < BT; ++T) {
      float f[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float z = zacc[T][r] + b1v;
        f[r] = z > 0.0f ? z : 0.0f;
      }
      uint32_t p[8];
      to_bf16x2(f, p);
#pragma unroll
      for (int r = 0; r < 16; ++r) a1[(32 * T + crow(r, lane)) * Ly::AS + n] = half_of(p, r);
      a1p[2 * T] = make_uint4(p[0], p[1], p[2], p[3]);
      a1p[2 * T + 1] = make_uint4(p[4], p[5], p[6], p[7]);
    }
    if (tid < BP) yl[tid] = ylab;
    __syncthreads();
    // ---- logits^T, softmax cross-entropy, argmax (lowest index on ties, a NaN
    //      logit is a miss), G2 = (p - onehot(y)) fl(1/b), or times the
    //      variant's per-element scale tensor when one is set.
    //      Up to 16 classes: 16-row batch tiles shared by all waves; a lane holds
    //      four classes of one row and the row's four lanes combine by shuffles.
    //      Classes 16..31 of G2 are then left unwritten and never read.
    //      More classes: one 32-row tile per wave; a lane holds the row's
    //      classes crow(r) of its half, combined with the other half.
    const bool c16 = a.C <= 16;
    if (c16) {
      const int l16 = lane & 15, lq = lane >> 4, C = a.C;
      for (int tt = wave; tt < BP / 16; tt += NW) {
        f32x4_t gsv = {scale, scale, scale, scale};   // the row's output-gradient scales (issued early)
        if (a.gscale) gsv = *reinterpret_cast<const f32x4_t*>(a.gscale + ((size_t)v * BP + 16 * tt + l16) * 32 + 4 * lq);
        f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
        const uint16_t* ap = w2 + l16 * Ly::W2S + 8 * lq;
        const uint16_t* bp = a1 + (16 * tt + l16) * Ly::AS + 8 * lq;
#pragma unroll
        for (int s = 0; s < HP / 32; ++s) acc = mma16(O::load(ap + 32 * s), O::load(bp + 32 * s), acc);
        const int b = 16 * tt + l16, y = yl[b];
        const bool rvalid = y >= 0;
        float z[4];
        float ml = -INFINITY, bv = -INFINITY;
        int bi = 64, nanl = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {                // j ascending = class ascending within the lane
          const int c = 4 * lq + j;
          z[j] = acc[j] + b2s[c];
          if (c < C) {
            ml = fmaxf(ml, z[j]);
            if (z[j] != z[j]) nanl = 1;
            else if (z[j] > bv) { bv = z[j]; bi = c; }
          }
        }
#pragma unroll
        for (int off = 16; off <= 32; off <<= 1) {
          ml = fmaxf(ml, __shfl_xor(ml, off));
          nanl |= __shfl_xor(nanl, off);
          const float ov = __shfl_xor(bv, off);
          const int oi = __shfl_xor(bi, off);
          if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
        }
        const float m = ml;
        float e[4], sl = 0.0f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          e[j] = 4 * lq + j < C ? expf(z[j] - m) : 0.0f;
          sl += e[j];
        }
        sl += __shfl_xor(sl, 16);                    // commutative pairings: the row's
        const float s = sl + __shfl_xor(sl, 32);     // four lanes hold the same sum
        float gf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = 4 * lq + j;
          gf[j] = (c < C && rvalid) ? (e[j] / s - (c == y ? 1.0f : 0.0f)) * gsv[j] : 0.0f;
        }
        uint32_t gq[2];
        to_bf16x2(gf, gq);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = 4 * lq + j;
          zg[c * Ly::ZGS + b] = gf[j];
          g2t[c * Ly::GTS + b] = half_of(gq, j);
          if (c == y) {                              // the label's lane records the row
            float ce = (logf(s) + m) - z[j];
            if (nanl) ce = NAN;
            rce[b] = (double)ce;
            rco[b] = (!nanl && bi == y) ? 1u : 0u;
          }
        }
        if (!rvalid && lq == 0) {
          rce[b] = 0.0;
          rco[b] = 0u;
        }
        *reinterpret_cast<uint2*>(g2 + b * Ly::GS + 4 * lq) = make_uint2(gq[0], gq[1]);
      }
    } else if (wave < BT) {
      f32x4_t gsv[4] = {{scale, scale, scale, scale}, {scale, scale, scale, scale}, {scale, scale, scale, scale},
                        {scale, scale, scale, scale}};   // classes 8q + 4lh + 0..3 of the row (issued early)
      if (a.gscale)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          gsv[q] = *reinterpret_cast<const f32x4_t*>(a.gscale + ((size_t)v * BP + 32 * wave + l32) * 32 + 8 * q + 4 * lh);
      f32x16_t c0 = zero16(), c1 = zero16();
      const uint16_t* ap = w2 + l32 * Ly::W2S + 8 * lh;
      const uint16_t* bp = a1 + (32 * wave + l32) * Ly::AS + 8 * lh;
#pragma unroll
      for (int s = 0; s < HP / 16; s += 2) {
        c0 = O::mma(O::load(ap + 16 * s), O::load(bp + 16 * s), c0);
        c1 = O::mma(O::load(ap + 16 * s + 16), O::load(bp + 16 * s + 16), c1);
      }
      const int b = 32 * wave + l32, C = a.C, y = yl[b];
      const bool rvalid = y >= 0;
      float z[16];
      float ml = -INFINITY, bv = -INFINITY;
      int bi = 64, nanl = 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) {                 // r ascending = class ascending within the lane
        const int c = crow(r, lane);
        z[r] = (c0[r] + c1[r]) + b2s[c];
        if (c < C) {
          ml = fmaxf(ml, z[r]);
          if (z[r] != z[r]) nanl = 1;
          else if (z[r] > bv) { bv = z[r]; bi = c; }
        }
      }
      const float m = fmaxf(ml, __shfl_xor(ml, 32));
      const int isn = nanl | __shfl_xor(nanl, 32);
      {
        const float ov = __shfl_xor(bv, 32);
        const int oi = __shfl_xor(bi, 32);
        if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
      }
      float e[16], sl = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        e[r] = crow(r, lane) < C ? expf(z[r] - m) : 0.0f;
        sl += e[r];
      }
      const float s = sl + __shfl_xor(sl, 32);       // same value in both halves
      float gf[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int c = crow(r, lane);
        gf[r] = (c < C && rvalid) ? (e[r] / s - (c == y ? 1.0f : 0.0f)) * gsv[r >> 2][r & 3] : 0.0f;
      }
      uint32_t gq[8];
      to_bf16x2(gf, gq);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int c = crow(r, lane);
        zg[c * Ly::ZGS + b] = gf[r];
        g2t[c * Ly::GTS + b] = half_of(gq, r);
        if (c == y) {                                // the label's lane records the row
          float ce = (logf(s) + m) - z[r];
          if (isn) ce = NAN;
          rce[b] = (double)ce;
          rco[b] = (!isn && bi == y) ? 1u : 0u;
        }
      }
      if (!rvalid && lh == 0) {
        rce[b] = 0.0;
        rco[b] = 0u;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<uint2*>(g2 + b * Ly::GS + 8 * q + 4 * lh) = make_uint2(gq[2 * q], gq[2 * q + 1]);
    }
    __syncthreads();
    // ---- db2 partial sums over row groups (fixed order); finished after the block loop
    {
      const int c = tid & 31, part = tid >> 5;       // Ly::NDP parts
      float sp = 0.0f;
      if (!c16 || c < 16)
        for (int r = part; r < BP; r += Ly::NDP) sp += zg[c * Ly::ZGS + r];
      dbp[part * 32 + c] = sp;
    }
    // the next pass's first blocks, W1 words and labels can load from here on
    // (the last step's pass also runs a forward, of a valid batch, whose result is unused)
    const int tf = t + 1 < a.T ? t + 1 : t;
    issue_head(on, t, on, tf, tid_step);
    // ---- dW2 = G2^T A1 (classes x hidden), A1 from registers
    f32x16_t d2 = zero16();
#pragma unroll
    for (int s = 0; s < NBS; ++s) {
      const uint16_t* pp = g2t + l32 * Ly::GTS + 16 * s + 4 * lh;
      d2 = O::mma(ld2x8(pp, pp + 8), a1p[s], d2);
    }
    // ---- G1 = (G2 W2) * ReLU' with the pre-update W2, taken from this lane's
    //      own master values (accumulators reuse zacc)
    float w2v[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 f = *reinterpret_cast<const float4*>(w2row + (((2 * q + lh) ^ sw) << 2));
      w2v[4 * q] = f.x; w2v[4 * q + 1] = f.y; w2v[4 * q + 2] = f.z; w2v[4 * q + 3] = f.w;
    }
    uint32_t pw2[8];
    to_bf16x2(w2v, pw2);
    const uint4 w2b[2] = {make_uint4(pw2[0], pw2[1], pw2[2], pw2[3]), make_uint4(pw2[4], pw2[5], pw2[6], pw2[7])};
#pragma unroll
    for (int T = 0; T < BT; ++T) {
      f32x16_t acc = zero16();
      {
        const uint16_t* pp = g2 + (32 * T + l32) * Ly::GS + 4 * lh;
        acc = O::mma(ld2x8(pp, pp + 8), w2b[0], acc);
      }
      if (!c16) {                                    // classes 16..31
        const uint16_t* pp = g2 + (32 * T + l32) * Ly::GS + 16 + 4 * lh;
        acc = O::mma(ld2x8(pp, pp + 8), w2b[1], acc);
      }
      zacc[T] = acc;
    }
    // ---- G1 operand slots (the A1 rows are no longer read) and db1
    float db1p = 0.0f;
#pragma unroll
    for (int T = 0; T < BT; ++T) {
      const uint32_t ap[8] = {a1p[2 * T].x, a1p[2 * T].y, a1p[2 * T].z, a1p[2 * T].w,
                              a1p[2 * T + 1].x, a1p[2 * T + 1].y, a1p[2 * T + 1].z, a1p[2 * T + 1].w};
      float f[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) f[r] = half_of(ap, r) != 0 ? zacc[T][r] : 0.0f;
      uint32_t p[8];
      to_bf16x2(f, p);
#pragma unroll
      for (int r = 0; r < 16; ++r) db1p += O::to_f32(half_of(p, r));
      g1s[(wave * NBS + 2 * T) * 64 + lane] = make_uint4(p[0], p[1], p[2], p[3]);
      g1s[(wave * NBS + 2 * T + 1) * 64 + lane] = make_uint4(p[4], p[5], p[6], p[7]);
    }
    db1p += __shfl_xor(db1p, 32);
    b1v = b1k ? __fsub_rn(b1v, __fmul_rn(lrv, db1p)) : 0.0f;
    // ---- masked SGD on W2 (LDS master) and refresh of its bf16 operand
    {
      float f[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) f[r] = ((m2bits >> r) & 1u) ? __fsub_rn(w2v[r], __fmul_rn(lrv2, d2[r])) : 0.0f;
      uint32_t p[8];
      to_bf16x2(f, p);
#pragma unroll
      for (int r = 0; r < 16; ++r) w2[crow(r, lane) * Ly::W2S + n] = half_of(p, r);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(w2row + (((2 * q + lh) ^ sw) << 2)) =
            make_float4(f[4 * q], f[4 * q + 1], f[4 * q + 2], f[4 * q + 3]);
    }
    // ---- dW1 + masked SGD on W1 + forward of the next step
    int tid_pass;
    asm volatile("v_mov_b32 %0, %1" : "=v"(tid_pass) : "v"(tid));
    kloop(on, t, on, tf, tid_pass);
  }
  __syncthreads();                             // the last step's partial sums
  finish_out();
  // ---- write back the resident state
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 f = *reinterpret_cast<const float4*>(w2row + (((2 * q + lh) ^ sw) << 2));
#pragma unroll
    for (int i = 0; i < 4; ++i) W2[((size_t)wave * 32 + crow(4 * q + i, lane)) * 32 + l32] = f4get(f, i);
  }
  if (lh == 0) a.b1[(size_t)v * HP + n] = b1v;
  if (tid < 32) a.b2[(size_t)v * 32 + tid] = b2s[tid];
  if (tid == tot_tid) {
    a.ce_acc[v] = ce_tot;
    a.correct_acc[v] = corr_tot;
  }
  vt_add(a.vtime, v, vt0);
}

size_t fused2_lds_bytes(int hp, int bp) {
  if (hp == 256 && bp == 128) return Fused2Lds<256, 128>::bytes;
  if (hp == 256 && bp == 64) return Fused2Lds<256, 64>::bytes;
  if (hp == 256 && bp == 32) return Fused2Lds<256, 32>::bytes;
  if (hp == 128 && bp == 128) return Fused2Lds<128, 128>::bytes;
  if (hp == 128 && bp == 64) return Fused2Lds<128, 64>::bytes;
  if (hp == 128 && bp == 32) return Fused2Lds<128, 32>::bytes;
  return 0;
}

template <int HP, int BP>
static hipError_t launch_f2(const Fused2Args& a, int P, hipStream_t s, const LaunchEv& ev) {
  static bool attr = false;
  const size_t lds = Fused2Lds<HP, BP>::bytes;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_fused2<HP, BP>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr = true;
  }
  hipExtLaunchKernelGGL((k_fused2<HP, BP>), dim3(P), dim3(2 * HP), lds, s, ev.start, ev.stop, 0, a);
  return hipGetLastError();
}

hipError_t launch_fused2(const Fused2Args& a, int P, hipStream_t s, const LaunchEv& ev) {
  if (a.Hp == 256 && a.Bp == 128) return launch_f2<256, 128>(a, P, s, ev);
  if (a.Hp == 256 && a.Bp == 64) return launch_f2<256, 64>(a, P, s, ev);
  if (a.Hp == 256 && a.Bp == 32) return launch_f2<256, 32>(a, P, s, ev);
  if (a.Hp == 128 && a.Bp == 128) return launch_f2<128, 128>(a, P, s, ev);
  if (a.Hp == 128 && a.Bp == 64) return launch_f2<128, 64>(a, P, s, ev);
  if (a.Hp == 128 && a.Bp == 32) return launch_f2<128, 32>(a, P, s, ev);
  return hipErrorInvalidValue;
}

}  // namespace gevo
