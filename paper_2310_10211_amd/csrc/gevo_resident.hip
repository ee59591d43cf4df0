// Resident training kernel for two-layer nets with 256 hidden units, a
// 128-row batch, 800 padded inputs and at most 16 classes (bf16 operands,
// fp32 masters; the update of paper section 6.2, fitness by retraining as in
// section 4.3).  A pair of workgroups trains one variant: each keeps the fp32
// master of the input weights of 128 hidden units on chip for the whole run
// (22 of the 25 32-column blocks in registers, the other 3 in LDS), so the
// masters cross memory once per run instead of twice per step.  The two
// halves meet once per step: each computes its units' share of the logits,
// the shares are swapped through memory, and both halves then take the
// identical softmax, loss and output gradient (the lower half's share is
// added first on both sides).
//
// Per step t (one wave per 32 hidden units, four waves per workgroup):
//   A1 = relu(Z1 + b1): rows -> LDS, bf16 pairs kept in registers
//   partial logits of this half -> exchange -> logits; softmax cross-entropy,
//     argmax (lowest index on ties, a NaN logit is a miss) and
//     G2 = (p - onehot(y)) fl(1/b) (or times the per-element scale tensor)
//   dW2 and G1 = (G2 W2) * ReLU' for this half's units (G1 stays in
//     registers as the operand of the next pass), db1, db2; W2, b1, b2 updated
//   pass 1, every 32-column block k:  dW1 = X_t^T G1,
//                                     W1 = mask ? fl(W1 - fl(lr dW1)) : +0
//   pass 2, every block k:            Z1' += X_{t+1} W1   (forward of step t+1)
// The accumulator layout of a 32x32 MFMA gives lane l the column l%32 and the
// rows 8(r/4) + 4(l/32) + r%4 of register r, and the eight registers 8s..8s+7
// of a tile serve as the operand of contraction step s.  That is how the W1
// registers (accumulators over the inputs of a block), G1 (over the batch)
// and A1 feed the MFMAs without leaving registers.  The other operand, X, is
// read from LDS in the matching order: the step's X copies are laid out with
// the middle two groups of four swapped within every 16 inputs (rows copy) or
// 16 batch rows (columns copy), so one 16-byte read gives a lane its eight
// operand elements.  X blocks reach LDS through direct-to-LDS loads into a
// ring of three blocks (two in flight), their 16-byte chunks XOR-swizzled
// against bank conflicts.  The loads are explicit instructions with explicit
// waits, so no compiler-inserted wait drains the ring.
//
// The exchange words carry the value and a step tag in one 64-bit word, so a
// reader polls its partner's words until every tag is current and needs no
// other ordering; the two parities alternate between steps, so a word is not
// rewritten before its reader is done with it.  The launch is cooperative
// (every workgroup resident at once), and a half that waits too long for its
// partner sets the error word and stops instead of hanging.
//
// Selected only on request (GEVO_RESIDENT=1): on gfx950 it is slower than the
// streaming fused kernel.  The 352 fp32 master values a lane keeps, with the
// accumulators and operands of a step, exceed what the register allocator
// places in the 256 VGPRs plus 256 AGPRs of a one-wave-per-SIMD workgroup; it
// spills about 1.7 KiB per lane to scratch, and the reloads (beyond L2 at
// this population size) sit in every block of the step.
#include "gevo_internal.h"
#include "gevo_device.h"

#include <math.h>

#include <type_traits>
#include <utility>

namespace gevo {

namespace {

constexpr int kW = 4;                    // waves per workgroup, 32 hidden units each
constexpr int kT = 64 * kW;              // threads
constexpr int kHC = 32 * kW;             // hidden units per workgroup
constexpr int kB = 128;                  // padded batch
constexpr int kBT = kB / 32;             // 32-row batch tiles
constexpr int kNBS = kB / 16;            // contraction steps over the batch
constexpr int kNKB = 25;                 // 32-column input blocks (800 padded inputs)
constexpr int kNR = 22;                  // blocks kept in registers
constexpr int kNL = kNKB - kNR;          // blocks kept in LDS
constexpr int kNS = 3;                   // X ring stages
constexpr int kJobs = 2 * kNKB;          // X blocks per step: pass 1, then pass 2
constexpr int kXBlk = kB * 32 * 2;       // bytes of one X block (rows or columns copy)
constexpr unsigned kMaxPoll = 1u << 20;  // exchange polls before a half gives up

static_assert(kResXW == kW * 2 * 64 * 4, "exchange words: 4 waves x 2 tiles x 64 lanes x 4 classes");

struct Lds {
  static constexpr int AS = kHC + 8;     // A1 rows [B][HC] and the W2 operand [16][HC]
  static constexpr int GS = 16 + 8;      // G2 rows [B][16]
  static constexpr int GTS = kB + 8;     // G2 columns [16][B]
  static constexpr int ZGS = kB + 1;     // fp32 G2 columns [16][B]
  static constexpr int NDP = kT / 16;    // db2 partial sums per class
  static constexpr size_t xr = 0;                                   // X ring [kNS][kXBlk]
  static constexpr size_t a1 = xr + (size_t)kNS * kXBlk;
  static constexpr size_t w2 = a1 + (size_t)kB * AS * 2;
  static constexpr size_t w2m = w2 + 16ull * AS * 2;                // fp32 master [HC][16], swizzled chunks
  static constexpr size_t g2 = w2m + (size_t)kHC * 16 * 4;
  static constexpr size_t g2t = g2 + (size_t)kB * GS * 2;
  static constexpr size_t zg = g2t + 16ull * GTS * 2;
  static constexpr size_t yl = zg + 16ull * ZGS * 4;
  static constexpr size_t b2 = yl + (size_t)kB * 4;
  static constexpr size_t dbp = b2 + 16 * 4;                        // [NDP][16]
  static constexpr size_t rce = (dbp + (size_t)NDP * 16 * 4 + 7) / 8 * 8;   // [B] fp64 per-row loss
  static constexpr size_t rco = rce + (size_t)kB * 8;               // [B] per-row hit
  static constexpr size_t w1l = (rco + (size_t)kB * 4 + 15) / 16 * 16;      // [kNL][kW][4][64] float4
  static constexpr size_t bytes = w1l + (size_t)kNL * kW * 4 * 64 * 16;
};
static_assert(Lds::bytes <= 160 * 1024, "LDS of the resident kernel");

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 ld2x8(const uint16_t* p0, const uint16_t* p1) {
  const uint2 lo = *reinterpret_cast<const uint2*>(p0);
  const uint2 hi = *reinterpret_cast<const uint2*>(p1);
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}

__device__ __forceinline__ uint16_t half_of(const uint32_t* p, int r) { return (uint16_t)(p[r >> 1] >> (16 * (r & 1))); }

// 16x16x32 bf16 MFMA: lane l supplies row (A) / column (B) l%16, contraction
// elements 8(l/16) .. 8(l/16)+7; the accumulator gives lane l the column l%16
// and the rows 4(l/16) .. 4(l/16)+3.
__device__ __forceinline__ f32x4_t mma16(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}


template <typename T>
__device__ __forceinline__ T* opaque_s(T* p) {
  asm volatile("" : "+s"(p));
  return p;
}

template <class F, int... J>
__device__ __forceinline__ void for_each_job(F&& f, std::integer_sequence<int, J...>) {
  (f(std::integral_constant<int, J>{}), ...);
}

}  // namespace

__global__ __launch_bounds__(kT, 1) void k_res2(Res2Args ra) {
  using O = Op<uint16_t>;
  const Fused2Args& a = ra.f;
  extern __shared__ __align__(16) char smem[];
  uint16_t* a1 = reinterpret_cast<uint16_t*>(smem + Lds::a1);
  uint16_t* w2 = reinterpret_cast<uint16_t*>(smem + Lds::w2);
  float* w2m = reinterpret_cast<float*>(smem + Lds::w2m);
  uint16_t* g2 = reinterpret_cast<uint16_t*>(smem + Lds::g2);
  uint16_t* g2t = reinterpret_cast<uint16_t*>(smem + Lds::g2t);
  float* zg = reinterpret_cast<float*>(smem + Lds::zg);
  int* yl = reinterpret_cast<int*>(smem + Lds::yl);
  float* b2s = reinterpret_cast<float*>(smem + Lds::b2);
  float* dbp = reinterpret_cast<float*>(smem + Lds::dbp);
  double* rce = reinterpret_cast<double*>(smem + Lds::rce);
  unsigned int* rco = reinterpret_cast<unsigned int*>(smem + Lds::rco);
  f32x4_t* w1l = reinterpret_cast<f32x4_t*>(smem + Lds::w1l);

  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, lh = lane >> 5, l16 = lane & 15, lq = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // workgroup -> (pair, half): with a multiple of 16 workgroups the two halves
  // of a pair are eight dispatch slots apart, i.e. on the same XCD
  const int G = gridDim.x, Q = G >> 1;
  int q, h;
  if (G % 16 == 0) {
    const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
    q = (j >> 1) * 8 + xcd;
    h = j & 1;
  } else {
    q = blockIdx.x >> 1;
    h = blockIdx.x & 1;
  }
  const int gw = kW * h + wave;                  // 32-unit block of the full hidden layer
  const int nl = wave * 32 + l32;                // this lane's unit within the half
  const int NWF = 2 * kW;                        // 32-unit blocks of the full layer
  const int HP = 2 * kHC;
  const int Kp = a.Kp;
  const size_t xstep = (size_t)Kp * kB * 2;      // bytes of one step's rows (or columns) copy
  const uint32_t ring = lds_addr(smem + Lds::xr);
  const int tot_tid = (kW - 1) * 64;             // thread that keeps the loss / hit totals

  // Direct-to-LDS lane offsets: instruction ii of this wave fills LDS chunks
  // P = 64 (2 wave + ii) + lane of a block.
  uint32_t cofs[2], rofs[2];
#pragma unroll
  for (int ii = 0; ii < 2; ++ii) {
    const int P = 64 * (2 * wave + ii) + lane;
    const int k = P >> 4, ck = (P & 15) ^ (k & 15);             // columns copy [32 inputs][B], 16 chunks a row
    cofs[ii] = (uint32_t)((k * kB + 8 * ck) * 2);
    const int b = P >> 2, cb = (P & 3) ^ ((b >> 2) & 3);        // rows copy [B][32 inputs], 4 chunks a row
    rofs[ii] = (uint32_t)((b * 32 + 8 * cb) * 2);
  }
  auto issue = [&](const char* base, size_t off, const uint32_t (&ofs)[2], int stage) {
    const char* blk = opaque_s(base) + off;      // the address of each block is formed where it is loaded
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
      dma16(blk, ofs[ii], ring + (uint32_t)(stage * kXBlk + (2 * wave + ii) * 1024));
  };
  const char* xrows = reinterpret_cast<const char*>(a.xrows);
  const char* xcols = reinterpret_cast<const char*>(a.xcols);

  f32x4_t wr[kNR][4];                            // W1 blocks 0..kNR-1 of this lane
  uint32_t mres[(kNKB + 1) / 2];                 // keep bits: block kb in half (kb & 1) of word kb / 2
  f32x16_t zacc[kBT];
  uint4 g1r[kNBS];
  bool failed = false;

  for (int v = q; v < ra.P && !failed; v += Q) {
    const uint64_t vt0 = vt_now();
    const int round = (v - q) / Q;
    float* W1 = a.W1 + (size_t)v * HP * Kp;
    const uint32_t* m1 = a.m1 + (size_t)v * HP * kNKB;
    float* W2 = a.W2 + (size_t)v * 32 * HP;
    const uint32_t* m2 = a.m2 + (size_t)v * 32 * NWF;
    const float lrv = a.lr[v];
    const float lrv2 = a.lr2 ? a.lr2[v] : lrv;   // output layer (the hidden layer's rate is 0 when removed)

    // ---- resident state of this half (register indices are compile-time constants)
    for_each_job(
        [&](auto kbc) {
          constexpr int kb = decltype(kbc)::value;
          const float* wp = W1 + ((size_t)kb * NWF + gw) * 1024 + lane * 4;
          const uint32_t word = m1[(size_t)kb * HP + gw * 32 + l32];
          uint32_t bits = 0;
#pragma unroll
          for (int r = 0; r < 16; ++r) bits |= ((word >> crow(r, lane)) & 1u) << r;
          if constexpr (kb % 2 == 0) mres[kb / 2] = bits;
          else mres[kb / 2] |= bits << 16;
#pragma unroll
          for (int qq = 0; qq < 4; ++qq) {
            const f32x4_t w = *reinterpret_cast<const f32x4_t*>(wp + qq * 256);
            if constexpr (kb < kNR) wr[kb][qq] = w;
            else w1l[(((kb - kNR) * kW + wave) * 4 + qq) * 64 + lane] = w;
          }
        },
        std::make_integer_sequence<int, kNKB>{});
    // output layer: this lane's 8 (class, unit) master values (classes
    // crow(r) for r < 8) in LDS row nl, 16-byte chunk c stored at
    // c ^ ((nl >> 2) & 3); bf16 operand copy [class][unit]; mask bits in a register
    float* w2row = w2m + nl * 16;
    const int sw = (nl >> 2) & 3;
    uint32_t m2bits = 0;
#pragma unroll
    for (int qq = 0; qq < 2; ++qq) {
      float f[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * qq + i, c = crow(r, lane);
        f[i] = W2[((size_t)gw * 32 + c) * 32 + l32];
        w2[c * Lds::AS + nl] = O::from_f32(f[i]);
        m2bits |= ((m2[c * NWF + gw] >> l32) & 1u) << r;
      }
      *reinterpret_cast<float4*>(w2row + (((2 * qq + lh) ^ sw) << 2)) = make_float4(f[0], f[1], f[2], f[3]);
    }
    if (tid < 16) b2s[tid] = a.b2[(size_t)v * 32 + tid];
    float b1v = a.b1[(size_t)v * HP + kHC * h + nl];
    const bool b1k = (a.bm1[(size_t)v * NWF + gw] >> l32) & 1u;
    const bool b2k = tid < 16 && ((a.bm2[v] >> (tid & 15)) & 1u);
    double ce_tot = 0.0;
    unsigned long long corr_tot = 0;
    if (h == 0 && tid == tot_tid) {
      ce_tot = a.ce_acc[v];
      corr_tot = a.correct_acc[v];
    }
    int ylab = -1;
    const int ylane = tid < kB ? tid : kB - 1;   // every thread loads (a uniform count of memory operations)

    // ---- pass 1 job (block kb of X_t^T): dW1, masked SGD of W1 block kb
    auto upd_block = [&](auto kbc, int stage, int ln) {
      constexpr int kb = decltype(kbc)::value;
      const int sw1 = (ln >> 5) ^ (ln & 15);       // chunk 2s + lh of row l32 is stored at 2s ^ sw1
      const char* xs = smem + Lds::xr + stage * kXBlk + 256 * (ln & 31);
      f32x16_t d = zero16();
#pragma unroll
      for (int s = 0; s < kNBS; ++s) {
        const uint4 xa = *reinterpret_cast<const uint4*>(xs + 16 * ((2 * s) ^ sw1));
        d = O::mma(xa, g1r[s], d);
      }
      uint32_t mb = mres[kb / 2] >> (16 * (kb % 2));
      asm volatile("" : "+v"(mb));              // keep bits read here, not hoisted as per-element conditions
      f32x4_t w[4];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        if constexpr (kb < kNR) w[qq] = wr[kb][qq];
        else w[qq] = w1l[(((kb - kNR) * kW + wave) * 4 + qq) * 64 + lane];
      }
      // masked SGD: the new value where the keep bit is set, +0 (all bits clear) elsewhere
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const uint32_t keep = (uint32_t)__builtin_amdgcn_sbfe((int)mb, r, 1);   // 0 or all ones
        w[r >> 2][r & 3] = __uint_as_float(__float_as_uint(__fsub_rn(w[r >> 2][r & 3], __fmul_rn(lrv, d[r]))) & keep);
      }
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        if constexpr (kb < kNR) wr[kb][qq] = w[qq];
        else w1l[(((kb - kNR) * kW + wave) * 4 + qq) * 64 + lane] = w[qq];
      }
    };
    // ---- pass 2 job (block kb of X rows): Z1 += X W1 block kb
    auto fwd_block = [&](auto kbc, int stage, int ln) {
      constexpr int kb = decltype(kbc)::value;
      const int l32 = ln & 31, lh = ln >> 5;
      const char* xs = smem + Lds::xr + stage * kXBlk;
      float f[16];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        f32x4_t w;
        if constexpr (kb < kNR) w = wr[kb][qq];
        else w = w1l[(((kb - kNR) * kW + wave) * 4 + qq) * 64 + lane];
#pragma unroll
        for (int i = 0; i < 4; ++i) f[4 * qq + i] = w[i];
      }
      uint32_t pw[8];
      to_bf16x2(f, pw);
      const uint4 wb[2] = {make_uint4(pw[0], pw[1], pw[2], pw[3]), make_uint4(pw[4], pw[5], pw[6], pw[7])};
#pragma unroll
      for (int T = 0; T < kBT; ++T) {
        const int b = 32 * T + l32;
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const uint4 xa = *reinterpret_cast<const uint4*>(xs + 64 * b + 16 * ((2 * s2 + lh) ^ ((b >> 2) & 3)));
          zacc[T] = O::mma(xa, wb[s2], zacc[T]);
        }
      }
    };

    // ---- forward of the first step (X rows of step t0, blocks issued two ahead)
    __syncthreads();                             // resident LDS state written
    {
      const char* xb = xrows + (size_t)a.t0 * xstep;
      issue(xb, 0, rofs, 0);
      issue(xb, kXBlk, rofs, 1);
      ylab = a.labels[(size_t)a.t0 * kB + ylane];
#pragma unroll
      for (int T = 0; T < kBT; ++T) zacc[T] = zero16();
      const int ln = opaque(lane);
      for_each_job(
          [&](auto jc) {
            constexpr int J = decltype(jc)::value;
            if constexpr (J == 0) wait_vm<3>();            // blocks 1 and the label may fly
            else if constexpr (J + 1 < kNKB) wait_vm<2>();
            else wait_vm<0>();
            __syncthreads();
            if constexpr (J + 2 < kNKB) issue(xb, (size_t)(J + 2) * kXBlk, rofs, (J + 2) % kNS);
            fwd_block(std::integral_constant<int, J>{}, J % kNS, ln);
          },
          std::make_integer_sequence<int, kNKB>{});
    }

    auto finish_out = [&]() {
      if (tid < 16) {
        float db = 0.0f;
#pragma unroll
        for (int part = 0; part < Lds::NDP; ++part) db += dbp[part * 16 + tid];
        b2s[tid] = b2k ? __fsub_rn(b2s[tid], __fmul_rn(lrv2, db)) : 0.0f;
      }
      if (wave == kW - 1) {
        double sc = 0.0;
        unsigned int co = 0;
        for (int r = lane; r < kB; r += 64) { sc += rce[r]; co += rco[r]; }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) { sc += __shfl_xor(sc, off); co += __shfl_xor(co, off); }
        if (lane == 0) { ce_tot += sc; corr_tot += co; }
      }
    };

    for (int t = a.t0; t < a.t1; ++t) {
      const int64_t r0 = (int64_t)t * a.B;
      const int bt = (int)((a.n - r0) < a.B ? (a.n - r0) : a.B);
      const float scale = __fdiv_rn(1.0f, (float)bt);
      const uint32_t cnt = (uint32_t)(round * (a.t1 - a.t0) + (t - a.t0) + 1);
      if (t > a.t0) finish_out();
      // ---- A1 = relu(Z1 + b1): rows -> LDS, bf16 operand pairs in registers
      uint4 a1p[kNBS];
#pragma unroll
      for (int T = 0; T < kBT; ++T) {
        float f[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float z = zacc[T][r] + b1v;
          f[r] = z > 0.0f ? z : 0.0f;
        }
        uint32_t p[8];
        to_bf16x2(f, p);
#pragma unroll
        for (int r = 0; r < 16; ++r) a1[(32 * T + crow(r, lane)) * Lds::AS + nl] = half_of(p, r);
        a1p[2 * T] = make_uint4(p[0], p[1], p[2], p[3]);
        a1p[2 * T + 1] = make_uint4(p[4], p[5], p[6], p[7]);
      }
      if (tid < kB) yl[tid] = ylab;
      __syncthreads();
      // ---- this half's share of the logits: 16-row batch tiles wave and wave + 4;
      //      a lane holds four classes of one row
      f32x4_t part[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int tt = wave + kW * i;
        f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
        const uint16_t* ap = w2 + l16 * Lds::AS + 8 * lq;
        const uint16_t* bp = a1 + (16 * tt + l16) * Lds::AS + 8 * lq;
#pragma unroll
        for (int s = 0; s < kHC / 32; ++s) acc = mma16(O::load(ap + 32 * s), O::load(bp + 32 * s), acc);
        part[i] = acc;
      }
      // ---- exchange with the other half
      {
        unsigned long long* own = ra.xbuf + (((size_t)q * 2 + h) * 2 + (cnt & 1u)) * kResXW;
        unsigned long long* oth = ra.xbuf + (((size_t)q * 2 + (h ^ 1)) * 2 + (cnt & 1u)) * kResXW;
        const size_t slot = (size_t)((wave * 2) * 64 + lane) * 4;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            __hip_atomic_store(own + slot + i * 256 + j,
                               ((unsigned long long)cnt << 32) | __float_as_uint(part[i][j]), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        f32x4_t other[2];
        unsigned int need = 0xffu, polls = 0;
        while (need != 0u && polls < kMaxPoll) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const unsigned long long x =
                  __hip_atomic_load(oth + slot + i * 256 + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              if ((uint32_t)(x >> 32) == cnt) {
                other[i][j] = __uint_as_float((uint32_t)x);
                need &= ~(1u << (4 * i + j));
              }
            }
          if (need != 0u) {
            ++polls;
            __builtin_amdgcn_s_sleep(1);
          }
        }
        if (__syncthreads_or(need != 0u)) {      // the partner did not answer: stop this workgroup
          if (tid == 0) __hip_atomic_store(ra.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          failed = true;
          break;
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) part[i][j] = h == 0 ? part[i][j] + other[i][j] : other[i][j] + part[i][j];
      }
      // ---- softmax cross-entropy, argmax and G2 (identical in both halves)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int tt = wave + kW * i, C = a.C;
        f32x4_t gsv = {scale, scale, scale, scale};
        if (a.gscale) gsv = *reinterpret_cast<const f32x4_t*>(a.gscale + ((size_t)v * kB + 16 * tt + l16) * 32 + 4 * lq);
        const int b = 16 * tt + l16, y = yl[b];
        const bool rvalid = y >= 0;
        float z[4];
        float ml = -INFINITY, bv = -INFINITY;
        int bi = 64, nanl = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {            // j ascending = class ascending within the lane
          const int c = 4 * lq + j;
          z[j] = part[i][j] + b2s[c];
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
        sl += __shfl_xor(sl, 16);                // commutative pairings: the row's
        const float s = sl + __shfl_xor(sl, 32); // four lanes hold the same sum
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
          zg[c * Lds::ZGS + b] = gf[j];
          g2t[c * Lds::GTS + b] = half_of(gq, j);
          if (c == y) {                          // the label's lane records the row
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
        *reinterpret_cast<uint2*>(g2 + b * Lds::GS + 4 * lq) = make_uint2(gq[0], gq[1]);
      }
      __syncthreads();
      // ---- db2 partial sums over row groups (fixed order); finished at the next step
      {
        const int c = tid & 15, pi = tid >> 4;
        float sp = 0.0f;
        for (int r = pi; r < kB; r += Lds::NDP) sp += zg[c * Lds::ZGS + r];
        dbp[pi * 16 + c] = sp;
      }
      // the first two X blocks of pass 1 and the labels of the next forward
      const int tf = t + 1 < a.T ? t + 1 : t;
      const char* xc = xcols + (size_t)t * xstep;
      const char* xn = xrows + (size_t)tf * xstep;
      issue(xc, 0, cofs, 0);
      issue(xc, kXBlk, cofs, 1);
      ylab = a.labels[(size_t)tf * kB + ylane];
      // ---- dW2 = G2^T A1 (classes x this half's units), A1 from registers
      f32x16_t d2 = zero16();
#pragma unroll
      for (int s = 0; s < kNBS; ++s) {
        const uint16_t* pp = g2t + l16 * Lds::GTS + 16 * s + 4 * lh;   // rows 16..31 of the tile are unused
        d2 = O::mma(ld2x8(pp, pp + 8), a1p[s], d2);
      }
      // ---- G1 = (G2 W2) * ReLU' with the pre-update W2 (this lane's master values)
      float w2v[8];
#pragma unroll
      for (int qq = 0; qq < 2; ++qq) {
        const float4 f = *reinterpret_cast<const float4*>(w2row + (((2 * qq + lh) ^ sw) << 2));
        w2v[4 * qq] = f.x; w2v[4 * qq + 1] = f.y; w2v[4 * qq + 2] = f.z; w2v[4 * qq + 3] = f.w;
      }
      uint32_t pw2[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pw2[i] = bf16x2(w2v[2 * i], w2v[2 * i + 1]);
      const uint4 w2b = make_uint4(pw2[0], pw2[1], pw2[2], pw2[3]);
      float db1p = 0.0f;
#pragma unroll
      for (int T = 0; T < kBT; ++T) {
        const uint16_t* pp = g2 + (32 * T + l32) * Lds::GS + 4 * lh;
        const f32x16_t acc = O::mma(ld2x8(pp, pp + 8), w2b, zero16());
        const uint32_t ap[8] = {a1p[2 * T].x, a1p[2 * T].y, a1p[2 * T].z, a1p[2 * T].w,
                                a1p[2 * T + 1].x, a1p[2 * T + 1].y, a1p[2 * T + 1].z, a1p[2 * T + 1].w};
        float f[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) f[r] = half_of(ap, r) != 0 ? acc[r] : 0.0f;
        uint32_t p[8];
        to_bf16x2(f, p);
#pragma unroll
        for (int r = 0; r < 16; ++r) db1p += O::to_f32(half_of(p, r));
        g1r[2 * T] = make_uint4(p[0], p[1], p[2], p[3]);
        g1r[2 * T + 1] = make_uint4(p[4], p[5], p[6], p[7]);
      }
      db1p += __shfl_xor(db1p, 32);
      b1v = b1k ? __fsub_rn(b1v, __fmul_rn(lrv, db1p)) : 0.0f;
      // ---- masked SGD on W2 (LDS master) and refresh of its bf16 operand
      {
        float f[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) f[r] = ((m2bits >> r) & 1u) ? __fsub_rn(w2v[r], __fmul_rn(lrv2, d2[r])) : 0.0f;
#pragma unroll
        for (int r = 0; r < 8; ++r) w2[crow(r, lane) * Lds::AS + nl] = O::from_f32(f[r]);
#pragma unroll
        for (int qq = 0; qq < 2; ++qq)
          *reinterpret_cast<float4*>(w2row + (((2 * qq + lh) ^ sw) << 2)) =
              make_float4(f[4 * qq], f[4 * qq + 1], f[4 * qq + 2], f[4 * qq + 3]);
      }
      // ---- pass 1 (dW1 + update), then pass 2 (forward of step tf), one X block per job
      const int ln1 = opaque(lane), ln2 = opaque(lane);
      for_each_job(
          [&](auto jc) {
            constexpr int J = decltype(jc)::value;
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (J == kNKB) {
#pragma unroll
              for (int T = 0; T < kBT; ++T) zacc[T] = zero16();
            }
            // in flight, in issue order: job 0, job 1, the labels; then two jobs ahead
            if constexpr (J <= 1) wait_vm<3>();
            else if constexpr (J + 1 < kJobs) wait_vm<2>();
            else wait_vm<0>();
            __syncthreads();
            if constexpr (J + 2 < kJobs) {
              constexpr int JN = J + 2;
              if constexpr (JN < kNKB) issue(xc, (size_t)JN * kXBlk, cofs, JN % kNS);
              else issue(xn, (size_t)(JN - kNKB) * kXBlk, rofs, JN % kNS);
            }
            if constexpr (J < kNKB) upd_block(std::integral_constant<int, J>{}, J % kNS, ln1);
            else fwd_block(std::integral_constant<int, J - kNKB>{}, J % kNS, ln2);
            __builtin_amdgcn_sched_barrier(0);
          },
          std::make_integer_sequence<int, kJobs>{});
    }
    if (failed) break;
    __syncthreads();                             // the last step's partial sums
    finish_out();
    __syncthreads();
    // ---- write back this half's state
    for_each_job(
        [&](auto kbc) {
          constexpr int kb = decltype(kbc)::value;
          float* wp = W1 + ((size_t)kb * NWF + gw) * 1024 + lane * 4;
#pragma unroll
          for (int qq = 0; qq < 4; ++qq) {
            f32x4_t w;
            if constexpr (kb < kNR) w = wr[kb][qq];
            else w = w1l[(((kb - kNR) * kW + wave) * 4 + qq) * 64 + lane];
            *reinterpret_cast<f32x4_t*>(wp + qq * 256) = w;
          }
        },
        std::make_integer_sequence<int, kNKB>{});
#pragma unroll
    for (int qq = 0; qq < 2; ++qq) {
      const float4 f = *reinterpret_cast<const float4*>(w2row + (((2 * qq + lh) ^ sw) << 2));
      const float fv[4] = {f.x, f.y, f.z, f.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) W2[((size_t)gw * 32 + crow(4 * qq + i, lane)) * 32 + l32] = fv[i];
    }
    if (lh == 0) a.b1[(size_t)v * HP + kHC * h + nl] = b1v;
    if (h == 0 && tid < 16) a.b2[(size_t)v * 32 + tid] = b2s[tid];
    if (h == 0 && tid == tot_tid) {
      a.ce_acc[v] = ce_tot;
      a.correct_acc[v] = corr_tot;
    }
    vt_add(a.vtime, v, vt0);
    __syncthreads();                             // LDS state of the next variant
  }
}

size_t res2_lds_bytes() { return Lds::bytes; }

bool res2_supported(int Kp, int Hp, int Bp, int C) { return Kp == 32 * kNKB && Hp == 2 * kHC && Bp == kB && C <= 16; }

int res2_max_pairs() {
  int dev = 0, ncu = 0, per_cu = 0, coop = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess || !coop) return 0;
  if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_res2), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)Lds::bytes);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(&k_res2), kT, Lds::bytes) !=
      hipSuccess)
    return 0;
  const int pairs = ncu * per_cu / 2;
  return pairs < kResMaxPairs ? pairs : kResMaxPairs;
}

hipError_t launch_res2(const Res2Args& a, int pairs, hipStream_t s, const LaunchEv& ev) {
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_res2), hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)Lds::bytes);
    attr = true;
  }
  if (!res2_supported(a.f.Kp, a.f.Hp, a.f.Bp, a.f.C) || pairs < 1 || pairs > kResMaxPairs) return hipErrorInvalidValue;
  if (ev.start) {
    const hipError_t e = hipEventRecord(ev.start, s);
    if (e != hipSuccess) return e;
  }
  Res2Args arg = a;
  void* args[] = {&arg};
  const hipError_t e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&k_res2), dim3(2 * pairs), dim3(kT),
                                                  args, (unsigned)Lds::bytes, s);
  if (e != hipSuccess) return e;
  if (ev.stop) return hipEventRecord(ev.stop, s);
  return hipSuccess;
}

}  // namespace gevo
