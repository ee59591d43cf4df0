// Prediction workload (paper section 4.3: a model is run over the dataset and
// its error recorded) for bf16 nets: every hidden layer of every variant is a
// plain GEMM over a chunk of test rows,
//   O_v = bf16(relu(A_v W_v + b_v)),
// with W_v a bf16 copy of the fp32 master rounded once per prediction call.
// When the last hidden layer is exactly one column tile wide, its GEMM also
// runs the output layer: logits, softmax cross-entropy, argmax (lowest index
// on ties, a NaN logit is a miss) and the tile's loss and hit sums, so the
// last hidden activations never leave the chip.
//
// One workgroup (eight waves, two per SIMD) computes a 256-row x 256-unit
// tile of one variant; the waves form a 4 x 2 grid of 64 x 128 tiles of
// 32x32x16 MFMAs (eight accumulator tiles per wave).  The contraction runs
// over 64-wide blocks (zero-filled past the input width) that reach LDS by
// direct-to-LDS loads, the input rows one block and the weights two blocks
// ahead of the multiply, so no registers stage them (two staging sets of
// registers left the waves, at 256 registers each, no room to read operand
// fragments ahead).
// Input rows and weights are both stored with
// the contraction index contiguous ([row][k] and [unit][k]), so both operand
// tiles load and read alike.  Workgroups that share a weight tile (same
// variant, all row tiles) run at the same time on one XCD (workgroup i runs
// on XCD i mod 8).
// One workgroup per CU runs its tiles back to back: the next tile's first
// operand blocks load while the finished tile is written out (or, with the
// output layer, while its logits and losses are formed), and the stores
// drain while the next tile computes (all CUs finish their tiles together,
// so a tile's 32 MB of output from the whole chip would otherwise be
// written, and the next workgroups dispatched, while no CU computes).
#include "gevo_internal.h"
#include "gevo_device.h"

#include <hip/hip_ext.h>
#include <math.h>

#include <type_traits>

namespace gevo {

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kPM = 256;                 // rows per tile
constexpr int kPN = 256;                 // units per tile
constexpr int kPK = 64;                  // contraction per block
constexpr int kPT = 512;                 // threads
// operand tile in LDS: 256 rows x 64 bf16, 128 B a row, 16-byte chunk c of
// row r stored at chunk c ^ ((r >> 1) & 7) (conflict-free operand reads)
constexpr size_t kTileBytes = (size_t)kPM * kPK * 2;
constexpr size_t kGemmLds = 5 * kTileBytes;            // two A buffers, then three W buffers (160 KiB)
// The epilogues use buffers 1 and 4 while the next tile's first blocks load
// into 0, 2 and 3.  Without the output layer each wave stages its rows in
// 8 KB of buffer 1 or 4; with it, buffer 1 holds the output layer's bf16
// operand [32 classes][kHS], its biases and the band sums, and buffer 4 the
// partial logits of the four row bands ([2][16][64] fp32 each).
constexpr int kHS = kPN + 8;
constexpr size_t kOutEnd = (size_t)32 * kHS * 2 + 32 * 4 + 4 * 8 + 4 * 4;
static_assert(kOutEnd <= kTileBytes && 4 * 2 * 16 * 64 * 4 <= kTileBytes, "epilogue scratch fits buffers 1 and 4");
static_assert(kGemmLds <= 160 * 1024, "LDS of one CU");

__device__ __forceinline__ f32x16_t mma32(u32x4_t a, u32x4_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}

}  // namespace

template <bool OUT>
__global__ __launch_bounds__(kPT, 1) void k_pred_gemm(PredGemmArgs a) {
  extern __shared__ __align__(16) char smem[];
  // Tiles: (variant, column tile) pairs p, each split into nr row tiles.
  // Workgroup b runs on XCD b % 8 and serves the pairs with p % 8 == b % 8,
  // row tile fastest: its s-th tile is tm = b / 8 + s * (gridDim.x / 8) of
  // that XCD's sequence, so the row tiles of a pair are in flight together on
  // one XCD and read its weight tile into that L2 once.  A launch holds one
  // workgroup per CU that runs its tiles back to back.
  const int nr = a.R / kPM, nn = a.Np / kPN, npairs = a.P * nn;
  const int xcd = blockIdx.x & 7, nwx = (int)(gridDim.x >> 3);
  const int cnt = xcd < npairs ? ((npairs - 1 - xcd) / 8 + 1) * nr : 0;   // tiles of this XCD
  int tm = (int)(blockIdx.x >> 3);
  if (tm >= cnt) return;
  int v, n0, r0, rt;
  auto set_tile = [&](int mm) {
    const int p = (mm / nr) * 8 + xcd;
    rt = mm % nr;
    v = p / nn;
    n0 = (p % nn) * kPN;
    r0 = rt * kPM;
  };
  set_tile(tm);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, lh = lane >> 5;
  const int wm = wave & 3, wn = wave >> 2;           // 64-row band, 128-unit band
  const int Kp = a.Kp;
  const int nblk = (Kp + kPK - 1) / kPK;
  const uint16_t* sA = a.A + a.a_vs * v + (size_t)r0 * Kp;
  const uint16_t* sW = a.W + ((size_t)v * a.Np + n0) * Kp;

  // Operand blocks go straight to LDS by direct-to-LDS loads: the input rows
  // (shared by all variants, mostly cache hits) one block ahead into two
  // buffers, the weights (first read from memory by the row tiles of a
  // variant) two blocks ahead into three.  Only waves 0-3 issue them: a
  // direct-to-LDS load waits at issue while the CU's load path is full (it
  // moves about 47 bytes a clock, so a block's 64 KB take ~1,400 of the
  // block's 2,048 MFMA clocks), and a wave waiting there issues no MFMA.
  // The matrix core of a SIMD serves its older wave first, so the younger
  // waves 4-7, which never wait there, fill it while waves 0-3 wait.
  // Loader wave w fills rows 64w .. 64w+63 of a tile, eight rows per
  // instruction: row group j = 8w + jj, lane l -> LDS chunk 64 j + l = row
  // 8 j + l / 8, stored chunk l % 8, which holds k chunk (l % 8) ^ ((row >>
  // 1) & 7).  Chunks past the input width are read from the row's first
  // chunk (in bounds) and zeroed in LDS once landed.
  const uint32_t lds0 = lds_addr(smem);
  const int wu = __builtin_amdgcn_readfirstlane(wave);   // the wave index as a scalar (LDS base in m0)
  const bool loader = wu < 4;
  const int lw = wave & 3;                               // loader rows (also set in waves 4-7, unused)
  uint32_t rowoff[8], cpos[8];
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) {
    const int r = 64 * lw + 8 * jj + (lane >> 3);
    rowoff[jj] = (uint32_t)r * (uint32_t)Kp * 2u;
    cpos[jj] = (uint32_t)((lane & 7) ^ ((r >> 1) & 7));   // k chunk this lane carries
  }
  auto abuf = [&](int kb) { return (size_t)(kb & 1) * kTileBytes; };
  auto wbuf = [&](int kb) { return (size_t)(2 + kb % 3) * kTileBytes; };
  auto issue = [&](const uint16_t* base, size_t buf, int kb, int j0 = 0, int j1 = 8) {
    if (!loader) return;
#pragma unroll
    for (int jj = j0; jj < j1; ++jj) {
      const int k = kb * kPK + 8 * (int)cpos[jj];
      const uint32_t voff = rowoff[jj] + (k < Kp ? (uint32_t)k * 2u : 0u);
      dma16(base, voff, lds0 + (uint32_t)buf + (uint32_t)((8 * wu + jj) * 1024));
    }
  };
  // after block kb's loads have landed: zero the loader lane's chunks past the input width
  auto zero_tail = [&](int kb) {
    if (loader && (kb + 1) * kPK > Kp) {
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
        if (kb * kPK + 8 * (int)cpos[jj] >= Kp) {
          const size_t at = (size_t)((8 * lw + jj) * 64 + lane) * 16;
          *reinterpret_cast<u32x4_t*>(smem + abuf(kb) + at) = u32x4_t{0u, 0u, 0u, 0u};
          *reinterpret_cast<u32x4_t*>(smem + wbuf(kb) + at) = u32x4_t{0u, 0u, 0u, 0u};
        }
    }
  };

  f32x16_t acc[2][4];

  // operand fragments of contraction step s (16 wide) of block kb: rows
  // wm*64 + 32i + l32 (A) and wn*128 + 32t + l32 (W), which all have
  // (row >> 1) & 7 == (l32 >> 1) & 7
  struct Frag {
    u32x4_t a[2], b[4];
  };
  auto rd = [&](Frag& f, int kb, int s) {
    // lane offsets formed at each read from an opaque lane id (hoisted out of
    // the loop they would hold a register per buffer and step)
    const int ln = opaque(lane), r32 = ln & 31;
    const char* as = smem + abuf(kb) + (size_t)(wm * 64 + r32) * 128;
    const char* ws = smem + wbuf(kb) + (size_t)(wn * 128 + r32) * 128;
    const int co = 16 * ((2 * s) ^ (ln >> 5) ^ ((r32 >> 1) & 7));
#pragma unroll
    for (int i = 0; i < 2; ++i) f.a[i] = *reinterpret_cast<const u32x4_t*>(as + i * 32 * 128 + co);
#pragma unroll
    for (int t = 0; t < 4; ++t) f.b[t] = *reinterpret_cast<const u32x4_t*>(ws + t * 32 * 128 + co);
  };
  auto mm = [&](const Frag& f) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[i][t] = mma32(f.b[t], f.a[i], acc[i][t]);
  };
  // The tile is accumulated transposed (units x rows): lane l holds row
  // wm*64 + 32i + l%32 and, in registers 4q..4q+3, the four consecutive
  // units wn*128 + 32t + 8q + 4(l/32) + 0..3.

  // a tile's first loads: A block 0, then W blocks 0 and 1 (eight loads each
  // in a loader wave), so a wait that leaves eight loads in flight covers
  // all but W block 1
  auto prologue = [&]() {
    int k0 = 0;
    asm volatile("" : "+s"(k0));                     // offsets formed here, not kept from the first tile
    issue(sA, abuf(k0), k0);
    issue(sW, wbuf(k0), k0);
    if (nblk > 1) issue(sW, wbuf(k0 + 1), k0 + 1);
  };
  // in place of A block nblk the tile's 256 biases go to LDS (one 1 KB
  // copy per wave, in the A buffer block nblk - 2 used)
  auto bias_to_lds = [&]() {
    dma16(a.bias + (size_t)v * a.Np + n0, (uint32_t)lane * 16u, lds0 + (uint32_t)abuf(nblk) + (uint32_t)wu * 1024u);
  };
  prologue();
  if (nblk > 1) wait_vm<8>();
  else wait_vm<0>();
  zero_tail(0);
  __syncthreads();
  for (;;) {
    const uint64_t vt0 = vt_now();
    asm volatile("" : : "s"(vt0));    // the clock read completes here, not pending in the loop
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[i][t] = zero16();
    // Fragments are read one contraction step ahead of the MFMAs that use
    // them, into two register sets.  Block kb's barrier sits before its last
    // step: by then every wave has read the whole block, so block kb + 1's
    // first fragments are read while the last step's MFMAs run.  Each step
    // also issues two of the wave's loads, one after its second and one after
    // its fifth MFMA: A block kb + 2 (into the A buffer block kb used) in
    // steps 3 and 0 after block kb's barrier, W block kb + 3 (into the W
    // buffer block kb used) in steps 1 and 2 of block kb + 1.  The last two
    // blocks are written out of the loop; scheduling fences keep this order.
    Frag f0, f1;
    struct Load {
      const uint16_t* base;
      size_t buf;
      int kb, j0;                                    // j0: a constant at every use
      bool on;
    };
    auto load1 = [&](const Load& l) {                // two of a loader wave's eight loads of a block
      if (l.on) issue(l.base, l.buf, l.kb, l.j0, l.j0 + 2);
    };
    auto mfma = [&](const Frag& f, int q) {
      const int i = q & 1, t = q >> 1;
      acc[i][t] = mma32(f.b[t], f.a[i], acc[i][t]);
    };
    auto step = [&](Frag& nxt, int kb_n, int s_n, const Frag& cur, const Load& l0, const Load& l1) {
      rd(nxt, kb_n, s_n);
      mfma(cur, 0);
      mfma(cur, 1);
      __builtin_amdgcn_sched_barrier(0);
      load1(l0);
      __builtin_amdgcn_sched_barrier(0);
      mfma(cur, 2);
      mfma(cur, 3);
      mfma(cur, 4);
      __builtin_amdgcn_sched_barrier(0);
      load1(l1);
      __builtin_amdgcn_sched_barrier(0);
      mfma(cur, 5);
      mfma(cur, 6);
      mfma(cur, 7);
      __builtin_amdgcn_sched_barrier(0);
    };
    const Load none{sA, 0, 0, 0, false};
    auto lA = [&](int j, int jj) { return Load{sA, abuf(j), j, jj, j < nblk}; };
    auto lW = [&](int j, int jj) { return Load{sW, wbuf(j), j, jj, j < nblk}; };
    // steps 0-2 of block kb (step 3's fragments read): the second half of
    // A block kb + 1, then W block kb + 2
    auto steps012 = [&](int kb) {
      step(f1, kb, 1, f0, lA(kb + 1, 4), lA(kb + 1, 6));
      step(f0, kb, 2, f1, lW(kb + 2, 0), lW(kb + 2, 2));
      step(f1, kb, 3, f0, lW(kb + 2, 4), lW(kb + 2, 6));
    };
    // the first half of A block 1 (or the biases) at the tile's start
    if (nblk > 1) issue(sA, abuf(1), 1, 0, 4);
    else bias_to_lds();
    rd(f0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    // (an opaque copy of nblk keeps the wait below in a block of its own, so
    // the compiler cannot sink the steps' MFMAs past the barrier)
    int nbo = nblk;
    asm volatile("" : "+s"(nbo));
    int kb = 0;
    for (; kb + 2 < nblk; ++kb) {
      steps012(kb);
      if (kb + 2 < nbo) wait_vm<8>();                // A and W block kb + 1 have landed
      else wait_vm<0>();
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
      step(f0, kb + 1, 0, f1, lA(kb + 2, 0), lA(kb + 2, 2));
    }
    if (kb + 1 < nblk) {                             // block nblk - 2
      steps012(kb);
      wait_vm<0>();
      zero_tail(kb + 1);
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
      bias_to_lds();
      step(f0, kb + 1, 0, f1, none, none);
      ++kb;
    }
    steps012(kb);                                    // block nblk - 1
    mm(f1);
    __builtin_amdgcn_sched_barrier(0);

    if constexpr (OUT) {
      // The layer is one tile wide (Np == 256): the tile holds whole rows of
      // the last hidden activation, and the output layer runs on it here.
      // H = bf16(relu(Z + b)) stays in registers as the operand of the
      // logits MFMAs: register 4q + e of accumulator (i, t) is unit
      // wn*128 + 32t + 8q + 4(l/32) + e of row wm*64 + 32i + l%32, so
      // registers 8s'..8s'+7 of (i, t) contract over the units
      // 32t + 16s' + {4(l/32) + 0..3, 8 + 4(l/32) + 0..3} of the wave's band,
      // and the output layer's bf16 weights are read from LDS in the same
      // order.  Each wave sums the logits over its 128 units; the two waves
      // of a row band add theirs in LDS.
      const size_t bslot = abuf(nblk) + (size_t)wave * 1024;
      wait_vm<0>();
      // lane-dependent offsets come from an opaque lane id, formed per tile
      // rather than held (and spilled) across the tile loop
      const int ln = opaque(lane), le32 = ln & 31, leh = ln >> 5;
      u32x4_t hf[2][4][2];
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 bn =
              *reinterpret_cast<const float4*>(smem + bslot + (size_t)(wn * 128 + t * 32 + 8 * q + 4 * leh) * 4);
          const float bv[4] = {bn.x, bn.y, bn.z, bn.w};
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            float f[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float z = acc[i][t][4 * q + e] + bv[e];
              f[e] = z > 0.0f ? z : 0.0f;
            }
            uint32_t pk[2];
            to_bf16x2(f, pk);
            hf[i][t][q >> 1][2 * (q & 1)] = pk[0];
            hf[i][t][q >> 1][2 * (q & 1) + 1] = pk[1];
          }
        }
      __syncthreads();                                   // every wave is done with the operand buffers
      // the output layer's operand [class][unit] (bf16) and biases into
      // buffer 1, the row labels of this wave's band into registers: every
      // load the compiler waits on completes before the next tile's
      // direct-to-LDS loads go out
      uint16_t* WL = reinterpret_cast<uint16_t*>(smem + kTileBytes);
      float* bL = reinterpret_cast<float*>(smem + kTileBytes + (size_t)32 * kHS * 2);
      double* red_ce = reinterpret_cast<double*>(smem + kTileBytes + (size_t)32 * kHS * 2 + 32 * 4);
      unsigned int* red_hit = reinterpret_cast<unsigned int*>(red_ce + 4);
      float* red = reinterpret_cast<float*>(smem + 4 * kTileBytes) + (size_t)wm * 2048;   // [2][16][64] per band
      {
        // master k-blocked [Np/32][32 classes][32 inputs]: thread tid converts
        // class tid / 8, inputs 32 (tid % 8) .. +31, half (tid >> 8)
        const float* WLm = a.WL + (size_t)v * 32 * kPN;
        const int c = (tid >> 3) & 31, kb = tid & 7, q0 = (tid >> 8) * 2;
        const float* src = WLm + ((size_t)kb * 32 + c) * 32;
#pragma unroll
        for (int q = q0; q < q0 + 2; ++q) {
          const float4 f0 = *reinterpret_cast<const float4*>(src + 8 * q);
          const float4 f1 = *reinterpret_cast<const float4*>(src + 8 * q + 4);
          const float f[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
          uint32_t pk[4];
          to_bf16x2(f, pk);
          *reinterpret_cast<u32x4_t*>(WL + c * kHS + kb * 32 + 8 * q) = u32x4_t{pk[0], pk[1], pk[2], pk[3]};
        }
        if (tid < 32) bL[tid] = a.bL[(size_t)v * 32 + tid];
      }
      int ylab[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) ylab[i] = a.labels[r0 + wm * 64 + 32 * i + le32];
      asm volatile("" : "+v"(ylab[0]), "+v"(ylab[1]));     // the label loads complete here
      __syncthreads();
      const int vcur = v, rtcur = rt;
      const bool more = tm + nwx < cnt;
      if (more) {                                        // the next tile's first blocks into buffers 0, 2, 3
        tm += nwx;
        set_tile(tm);
        sA = a.A + a.a_vs * v + (size_t)r0 * Kp;
        sW = a.W + ((size_t)v * a.Np + n0) * Kp;
        prologue();
      }
      f32x16_t lg[2] = {zero16(), zero16()};
      {
        const uint16_t* wrow = WL + le32 * kHS + wn * 128 + 4 * leh;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2) {
            const uint2 lo = *reinterpret_cast<const uint2*>(wrow + 32 * t + 16 * s2);
            const uint2 hi = *reinterpret_cast<const uint2*>(wrow + 32 * t + 16 * s2 + 8);
            const u32x4_t wf = u32x4_t{lo.x, lo.y, hi.x, hi.y};
#pragma unroll
            for (int i = 0; i < 2; ++i) lg[i] = mma32(wf, hf[i][t][s2], lg[i]);
          }
      }
      if (wn == 1) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) red[(i * 16 + r) * 64 + ln] = lg[i][r];
      }
      __syncthreads();
      if (wn == 0) {
        // logits^T of the band's rows: lane holds row 32i + l32 and classes
        // crow(r) of its half; the row's other half is in lane ^ 32
        const int C = a.C;
        double ce_sum = 0.0;
        unsigned int hits = 0;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int y = ylab[i];
          float z[16];
          float m = -INFINITY, bv = -INFINITY;
          int bi = 64, nanl = 0;
#pragma unroll
          for (int r = 0; r < 16; ++r) {               // r ascending = class ascending within the lane
            const int c = crow(r, ln);
            z[r] = (lg[i][r] + red[(i * 16 + r) * 64 + ln]) + bL[c];
            if (c < C) {
              m = fmaxf(m, z[r]);
              if (z[r] != z[r]) nanl = 1;
              else if (z[r] > bv) { bv = z[r]; bi = c; }
            }
          }
          m = fmaxf(m, __shfl_xor(m, 32));
          nanl |= __shfl_xor(nanl, 32);
          {
            const float ov = __shfl_xor(bv, 32);
            const int oi = __shfl_xor(bi, 32);
            if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
          }
          float sl = 0.0f, zy = 0.0f;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int c = crow(r, ln);
            if (c < C) sl += expf(z[r] - m);
            if (c == y) zy = z[r];
          }
          const float s = sl + __shfl_xor(sl, 32);
          zy += __shfl_xor(zy, 32);                    // exactly one lane of the pair holds class y
          float ce = (logf(s) + m) - zy;
          if (nanl) ce = NAN;
          if (leh == 0 && y >= 0) {
            ce_sum += (double)ce;
            hits += (!nanl && bi == y) ? 1u : 0u;
          }
        }
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) {      // lanes 0..31 hold the rows; fixed order
          ce_sum += __shfl_xor(ce_sum, off);
          hits += __shfl_xor(hits, off);
        }
        if (lane == 0) { red_ce[wm] = ce_sum; red_hit[wm] = hits; }
      }
      __syncthreads();
      if (tid == 0) {
        double t = 0.0;
        unsigned int hsum = 0;
        for (int w = 0; w < 4; ++w) { t += red_ce[w]; hsum += red_hit[w]; }
        a.part_ce[(size_t)vcur * a.n_chunks_total + a.chunk0 + rtcur] = t;
        a.part_correct[(size_t)vcur * a.n_chunks_total + a.chunk0 + rtcur] = hsum;
      }
      vt_add(a.vtime, vcur, vt0);
      if (!more) return;
      // the next tile's A and W block 0 have landed (W block 1 and this
      // tile's last stores may stay in flight)
      if (nblk > 1) wait_vm<8>();
      else wait_vm<0>();
      zero_tail(0);
      __syncthreads();
    } else {
      // The tile's biases (in LDS since the last block began) are added to
      // the accumulators (lane: units wn*128 + 32t + 8q + 4(l/32) + 0..3);
      // no load that the compiler waits on is ever in flight.
      const size_t bslot = abuf(nblk) + (size_t)wave * 1024;
      wait_vm<0>();
      // lane-dependent offsets of the write-out come from an opaque lane id,
      // formed per tile rather than held across the tile loop
      const int ln = opaque(lane), le32 = ln & 31, leh = ln >> 5;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 bn =
              *reinterpret_cast<const float4*>(smem + bslot + (size_t)(wn * 128 + t * 32 + 8 * q + 4 * leh) * 4);
          const float bv[4] = {bn.x, bn.y, bn.z, bn.w};
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[i][t][4 * q + e] = acc[i][t][4 * q + e] + bv[e];
        }
      __syncthreads();                                 // every wave is done with the operand buffers
      uint16_t* Out = a.O + a.o_vs * v + (size_t)r0 * a.Np + n0;
      const int vdone = v;
      // The next tile's first blocks load into buffers 0, 2 and 3 while this
      // tile is written out through buffers 1 and 4.
      const bool more = tm + nwx < cnt;
      if (more) {
        tm += nwx;
        set_tile(tm);
        sA = a.A + a.a_vs * v + (size_t)r0 * Kp;
        sW = a.W + ((size_t)v * a.Np + n0) * Kp;
        prologue();
      }
      // ReLU -> bf16 -> global rows, per wave in two rounds of 64 rows x 64
      // units staged in the wave's own 8 KB of LDS (16-byte chunk c of row r
      // at c ^ (r & 7)), then read back as whole 128-byte row segments: eight
      // rows per store instruction, sixteen store instructions per wave.
      char* st = smem + (size_t)(wn ? 4 : 1) * kTileBytes + (size_t)wm * 8192;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int i = 0; i < 2; ++i) {
              const int row = 32 * i + le32, c = 4 * tt + q;
              float f[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float z = acc[i][2 * h + tt][4 * q + e];
                f[e] = z > 0.0f ? z : 0.0f;
              }
              uint32_t pk[2];
              to_bf16x2(f, pk);
              *reinterpret_cast<uint2*>(st + row * 128 + ((c ^ (row & 7)) << 4) + (leh << 3)) = make_uint2(pk[0], pk[1]);
            }
#pragma unroll
        for (int it = 0; it < 8; ++it) {
          const int row = 8 * it + (ln >> 3), c = ln & 7;
          const u32x4_t val = *reinterpret_cast<const u32x4_t*>(st + row * 128 + ((c ^ (row & 7)) << 4));
          __builtin_nontemporal_store(val, reinterpret_cast<u32x4_t*>(Out + (size_t)(wm * 64 + row) * a.Np +
                                                                      wn * 128 + 64 * h + 8 * c));
        }
      }
      vt_add(a.vtime, vdone, vt0);
      if (!more) return;
      // every memory operation after the next tile's first weight block (its
      // second weight block, then at least the sixteen stores) may stay in flight
      if (nblk > 1) wait_vm<24>();
      else wait_vm<16>();
      zero_tail(0);
      __syncthreads();
    }
  }
}

// bf16 operand copy of a hidden layer's master: from the k-blocked fp32
// master [P][Kp/32][Np][32] to [P][Np][Kp], one workgroup per (variant,
// 32-input block, 256 units); thread t converts unit t's 32 inputs.
__global__ __launch_bounds__(256) void k_wt_bf16(const float* __restrict__ Wm, uint16_t* __restrict__ Wb, int Kp,
                                                 int Np) {
  const int nkb = Kp / 32, ntile = Np / 256;
  const int64_t b = blockIdx.x;
  const int v = (int)(b / ((int64_t)nkb * ntile)), rem = (int)(b % ((int64_t)nkb * ntile));
  const int kb = rem / ntile, n = (rem % ntile) * 256 + threadIdx.x;
  const float* src = Wm + (((size_t)v * nkb + kb) * Np + n) * 32;
  uint16_t* dst = Wb + ((size_t)v * Np + n) * Kp + kb * 32;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 f0 = *reinterpret_cast<const float4*>(src + 8 * q);
    const float4 f1 = *reinterpret_cast<const float4*>(src + 8 * q + 4);
    const float f[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
    uint32_t pk[4];
    to_bf16x2(f, pk);
    *reinterpret_cast<u32x4_t*>(dst + 8 * q) = u32x4_t{pk[0], pk[1], pk[2], pk[3]};
  }
}

bool pred_gemm_supported(int Kp, int Np, int R) {
  return Kp % 32 == 0 && Kp > 0 && Np % kPN == 0 && R % kPM == 0 && R > 0;
}

hipError_t launch_wt_bf16(const float* Wm, uint16_t* Wb, int P, int Kp, int Np, hipStream_t s, const LaunchEv& ev) {
  if (Kp % 32 || Np % 256 || P <= 0) return hipErrorInvalidValue;
  const int64_t blocks = (int64_t)P * (Kp / 32) * (Np / 256);
  hipExtLaunchKernelGGL(k_wt_bf16, dim3((unsigned)blocks), dim3(256), 0, s, ev.start, ev.stop, 0, Wm, Wb, Kp, Np);
  return hipGetLastError();
}

// compute units of the current device, cached per device
static int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cus[dev] = n;
  }
  return cus[dev];
}

template <bool OUT>
static hipError_t launch_pg(const PredGemmArgs& a, hipStream_t s, const LaunchEv& ev) {
  constexpr size_t lds = kGemmLds;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pred_gemm<OUT>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr = true;
  }
  const int64_t pairs = (int64_t)a.P * (a.Np / kPN);
  int64_t per_xcd = (pairs + 7) / 8 * (a.R / kPM);      // tiles of the busiest XCD
  const int cus = device_cus();                          // one workgroup per CU, tiles back to back
  if (cus < 8) return hipErrorInvalidDevice;
  if (per_xcd > cus / 8) per_xcd = cus / 8;
  hipExtLaunchKernelGGL((k_pred_gemm<OUT>), dim3((unsigned)(8 * per_xcd)), dim3(kPT), lds, s, ev.start, ev.stop, 0,
                        a);
  return hipGetLastError();
}

hipError_t launch_pred_gemm(const PredGemmArgs& a, hipStream_t s, const LaunchEv& ev) {
  if (!pred_gemm_supported(a.Kp, a.Np, a.R)) return hipErrorInvalidValue;
  if (a.WL) {
    if (a.Np != kPN || a.C < 1 || a.C > 32 || !a.bL || !a.labels || !a.part_ce || !a.part_correct)
      return hipErrorInvalidValue;
    return launch_pg<true>(a, s, ev);
  }
  return launch_pg<false>(a, s, ev);
}

}  // namespace gevo
