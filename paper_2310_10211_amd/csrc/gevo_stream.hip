// Hidden layer of a deeper bf16 net for one SGD step (section 6.2: the mean
// output gradient times the learning rate updates weights and biases;
// section 4.3: fitness by retraining), fused with the forward of the next
// step, for variant v and 128 of the layer's units:
//   dW[k][n] = sum_b A_t[b][k] G[b][n]                  (MFMA, contraction = batch)
//   W        = mask ? fl(W - fl(lr dW)) : +0          (fp32 master, in place)
//   b        = bmask ? fl(b - fl(lr sum_b G[b][n])) : +0
//   Z[b][n]  = sum_k A_{t+1}[b][k] bf16(W)[k][n] + b,  O = bf16(relu(Z))
//
// The fp32 master streams once per step, 32 inputs (one k-block) at a time,
// through registers, in the register-image layout (each load or store of a
// wave moves one contiguous KiB; the launcher keeps that copy of the master
// and its block-major mask words current).  Four waves, one per SIMD with the
// whole register file:
// wave w owns units 32w..32w+31.  For a block, the weight gradient comes out
// of 32x32x16 MFMAs in the accumulator layout (lane l: unit l%32, inputs
// k = 8(r/4) + 4(l/32) + r%4 of register r), is applied in place, rounded to
// bf16 and used at once as the B operand of the next step's forward; the A
// operand (input rows) is read from LDS in the same k order, so the
// contraction pairs every product correctly.  The gradient G stays in
// registers for the whole pass; the input blocks of both orientations are
// staged through LDS (two buffers); the master is prefetched two blocks ahead
// with explicit loads and explicit waits (checked on the assembly at build
// time).
#include "gevo_internal.h"
#include "gevo_device.h"

#include <hip/hip_ext.h>

#include <type_traits>

namespace gevo {

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kSU = 128;                 // units per workgroup
constexpr int kSW = 4;                   // waves per workgroup
constexpr int kST = 64 * kSW;

__device__ __forceinline__ f32x16_t mma32(u32x4_t a, u32x4_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}

template <int BP>
struct StreamLds {                       // sizes in bf16 elements, two buffers of each
  // input rows of a block [BP][32]: an 18-dword row stride puts the 32 rows
  // of an 8-byte fragment read on distinct bank pairs
  static constexpr int XR = 36;
  static constexpr int XC = BP + 8;      // input columns of a block [32][BP]
  static constexpr int rows = BP * XR;
  static constexpr int cols = 32 * XC;
  // per wave, the block's transposed operand copy [32 k][32 n] on its way to
  // global memory; a 40-element (80-byte) row stride puts the rows k and
  // k + 4 that one 2-byte write instruction touches on different banks
  static constexpr int TR = 40;
  static constexpr int tcopy = kSW * 32 * TR;
  static constexpr size_t bytes = ((size_t)2 * (rows + cols) + tcopy) * 2;
};

}  // namespace

template <int BP, bool UPD, bool FWD>
__global__ __launch_bounds__(kST, 1) void k_stream_layer(LayerArgs<uint16_t> a) {
  typedef StreamLds<BP> Ly;
  constexpr int NBS = BP / 16;           // contraction steps of the update
  constexpr int BT = BP / 32;            // 32-row forward tiles
  constexpr int XU = BP / 64;            // 16-byte chunks per thread per block and orientation
  constexpr int NX = (UPD ? XU : 0) + (FWD ? XU : 0);
  constexpr int NW = UPD ? 5 : 4;        // vector memory operations of one master block (+ its mask word)
  constexpr int S = UPD ? 4 : 0;         // master stores of one block (transposed-copy stores follow them)
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* xr = lds;
  uint16_t* xc = lds + 2 * Ly::rows;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, lh = lane >> 5;
  uint16_t* tw = lds + 2 * (Ly::rows + Ly::cols) + wave * 32 * Ly::TR;   // this wave's transpose tile
  // the tiles of one variant share an XCD and its L2 (workgroup i runs on XCD i % 8)
  int v, tile;
  {
    const int gx = gridDim.x, total = gx * gridDim.y, i = blockIdx.y * gx + blockIdx.x;
    const int j = total % 8 == 0 ? (i % 8) * (total / 8) + i / 8 : i;
    v = j / gx;
    tile = j % gx;
  }
  const uint64_t vt0 = vt_now();
  if (a.wout && tile * kSU >= (int)a.wout[v]) {         // every unit of the tile removed
    vt_add(a.vtime, v, vt0);
    return;
  }
  const int Kp = a.Kp, Np = a.Np, nkb = Kp / 32, last = nkb - 1;
  // Each tile visits the k-blocks in its own rotated order, so that the
  // workgroups streaming at the same time read different lines of a shared
  // input rather than all the same ones (visit j is block phys(j)).
  const int rot = (v * (int)gridDim.x + tile) % nkb;
  auto phys = [&](int j) { return j + rot < nkb ? j + rot : j + rot - nkb; };
  const int n = tile * kSU + wave * 32 + l32;          // this lane's unit
  const float lrv = a.lr[v];
  // Scalar bases of the master image and mask words (see below).  Declared
  // here, before the gradient loads, the compiler keeps them in scalar
  // registers; the build rejects a base in vector registers (the assembler)
  // or one moved there from vector registers (check_prefetch.sgpr_hazards).
  float* wimg = a.Wimg + (size_t)v * Np * Kp;
  const uint32_t* mblk = a.mblk + (size_t)v * nkb * Np;

  // the gradient at this layer's output for the whole pass: gs[s] holds
  // G[n][16s + 8lh .. +7], the B operand of contraction step s
  u32x4_t gs[UPD ? NBS : 1];
  float bias_n;
  {
    float db = 0.0f;
    if constexpr (UPD) {
      const uint16_t* gp = a.Gcols + a.g_vs * v + (size_t)n * BP + 8 * lh;
#pragma unroll
      for (int s = 0; s < NBS; ++s) {
        gs[s] = *reinterpret_cast<const u32x4_t*>(gp + 16 * s);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          db += bf16_bits_to_f32((uint16_t)gs[s][i]) + bf16_bits_to_f32((uint16_t)(gs[s][i] >> 16));
      }
      db += __shfl_xor(db, 32);                        // the other half of the batch
    }
    const float bo = a.bias[(size_t)v * Np + n];
    const bool bk = (a.bmask[(size_t)v * (Np / 32) + n / 32] >> (n % 32)) & 1u;
    bias_n = UPD ? (bk ? __fsub_rn(bo, __fmul_rn(lrv, db)) : 0.0f) : bo;
  }

  // Loads take a uniform base (scalar registers, block-dependent) plus a
  // loop-invariant 32-bit lane offset in bytes.
  const uint16_t* acol = UPD ? a.Acols + a.ac_vs * v : nullptr;   // [Kp][BP]
  const uint16_t* arow = FWD ? a.Arows + a.ar_vs * v : nullptr;   // [BP][Kp]
  // master image of this variant: block kb, unit group g (32 units) holds
  // 4 KiB as [q][lane][4], lane l32 + 32lh holding inputs 8q + 4lh + 0..3 of
  // unit 32g + l32; mask words block-major [kb][n].  The scalar base of a
  // block depends on the variant and the block only; the unit group goes
  // into the 32-bit lane offset, so no base is ever moved from a vector
  // register (a VALU write of an SGPR that a memory instruction reads needs
  // five wait states, which the compiler does not insert before inline
  // assembly).
  uint32_t oc[XU], orr[XU];
#pragma unroll
  for (int q = 0; q < XU; ++q) {
    const int i = tid + kST * q;
    oc[q] = (uint32_t)(((i / (BP / 8)) * BP + (i % (BP / 8)) * 8) * 2);
    orr[q] = (uint32_t)(((i >> 2) * Kp + (i & 3) * 8) * 2);
  }
  const int grp = tile * (kSU / 32) + wave;            // this wave's 32-unit group
  const uint32_t ow = (uint32_t)((grp * 1024 + lane * 4) * 4), om = (uint32_t)(n * 4);
  // input staging, two register sets used alternately by even and odd
  // visits: columns in [0, XU), rows in [XU, 2XU)
  u32x4_t stE[2 * XU], stO[2 * XU];
  // staging load i (0 <= i < NX: the column loads, then the row loads) of
  // visit j: columns of visit j + 2, rows of visit j + 1 (clamped to the last
  // visit, re-read in bounds and never used)
  auto load_x1 = [&](int j, int i, u32x4_t (&st)[2 * XU]) {
    const int jc = min(j + 2, last), jr = min(j + 1, last);
    if (UPD && i < XU) {
      const uint16_t* bc = acol + (size_t)phys(jc) * 32 * BP;
      asm volatile("global_load_dwordx4 %0, %1, %2" : "=&v"(st[i]) : "v"(oc[i]), "s"(bc) : "memory");
    } else if constexpr (FWD) {
      const int q = UPD ? i - XU : i;
      const uint16_t* br = arow + phys(jr) * 32;
      asm volatile("global_load_dwordx4 %0, %1, %2" : "=&v"(st[XU + q]) : "v"(orr[q]), "s"(br) : "memory");
    }
  };
  auto store_xc = [&](int buf, const u32x4_t (&st)[2 * XU]) {
    if constexpr (UPD) {
#pragma unroll
      for (int q = 0; q < XU; ++q) {
        const int i = tid + kST * q;
        *reinterpret_cast<u32x4_t*>(xc + buf * Ly::cols + (i / (BP / 8)) * Ly::XC + (i % (BP / 8)) * 8) = st[q];
      }
    }
  };
  auto store_xr = [&](int buf, const u32x4_t (&st)[2 * XU]) {
    if constexpr (FWD) {
#pragma unroll
      for (int q = 0; q < XU; ++q) {
        const int i = tid + kST * q;
        uint16_t* d = xr + buf * Ly::rows + (i >> 2) * Ly::XR + (i & 3) * 8;   // 8-byte aligned rows
        *reinterpret_cast<u32x2_t*>(d) = u32x2_t{st[XU + q][0], st[XU + q][1]};
        *reinterpret_cast<u32x2_t*>(d + 4) = u32x2_t{st[XU + q][2], st[XU + q][3]};
      }
    }
  };
  // this lane's master values of block kb: k = 32kb + 8q + 4lh + 0..3
  // (q = 0..3: one contiguous KiB of the wave's image per load), and the
  // unit's mask word
  auto load_w = [&](int j, f32x4_t (&w)[4], uint32_t& m) {
    const int kb = phys(j);
    const float* bw = wimg + (size_t)kb * Np * 32;     // the block's image: Np/32 groups of 1024 floats
    if constexpr (UPD) {
      const uint32_t* bm = mblk + (size_t)kb * Np;
      asm volatile(
          "global_load_dwordx4 %0, %5, %6\n\t"
          "global_load_dwordx4 %1, %5, %6 offset:1024\n\t"
          "global_load_dwordx4 %2, %5, %6 offset:2048\n\t"
          "global_load_dwordx4 %3, %5, %6 offset:3072\n\t"
          "global_load_dword %4, %7, %8"
          : "=&v"(w[0]), "=&v"(w[1]), "=&v"(w[2]), "=&v"(w[3]), "=&v"(m)
          : "v"(ow), "s"(bw), "v"(om), "s"(bm)
          : "memory");
    } else {
      asm volatile(
          "global_load_dwordx4 %0, %4, %5\n\t"
          "global_load_dwordx4 %1, %4, %5 offset:1024\n\t"
          "global_load_dwordx4 %2, %4, %5 offset:2048\n\t"
          "global_load_dwordx4 %3, %4, %5 offset:3072"
          : "=&v"(w[0]), "=&v"(w[1]), "=&v"(w[2]), "=&v"(w[3])
          : "v"(ow), "s"(bw)
          : "memory");
      m = 0u;
    }
  };

  f32x16_t z[BT];
#pragma unroll
  for (int T = 0; T < BT; ++T) z[T] = zero16();
  uint32_t pp[8];                                      // bf16 B operand of the previous visit

  // forward of the previous visit's block: rows 32T + l32 from buffer buf,
  // k = 16s2 + 4lh + {0..3, 8..11}, B operand from pp
  auto forward = [&](int buf) {
    const uint16_t* xrb = xr + buf * Ly::rows + l32 * Ly::XR + 4 * lh;
    u32x4_t xf[2 * BT];
#pragma unroll
    for (int i = 0; i < 2 * BT; ++i) {
      const uint16_t* p = xrb + 32 * (i >> 1) * Ly::XR + 16 * (i & 1);
      const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(p);
      const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(p + 8);
      xf[i] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
    }
    const u32x4_t wb[2] = {{pp[0], pp[1], pp[2], pp[3]}, {pp[4], pp[5], pp[6], pp[7]}};
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int T = 0; T < BT; ++T) z[T] = mma32(xf[2 * T + s2], wb[s2], z[T]);
  };

  // Visit j: the weight gradient of block phys(j) (inputs in column buffer
  // j&1) with visit j's staging loads (columns of j+2, rows of j+1, into the
  // register set of j's parity) spread between its MFMAs, the forward of
  // visit j-1 (rows in buffer (j-1)&1) while the update of visit j is
  // applied, the master stores of j and the master words of j+2 into the
  // registers just consumed, then visit j-1's staged inputs (columns of j+1,
  // rows of j) into LDS and a barrier.  Vector memory operations retire in
  // issue order.  Younger than visit j's master words (issued by visit j-2)
  // are visit j-1's staging loads (NX), master stores (S) and master words
  // of j+1 (NW); younger than visit j-1's staging loads are visit j-1's
  // stores and master words and visit j's staging loads, stores and master
  // words.  (Younger transposed-copy stores only make a wait stricter.)
  // For visit 0 the prologue issued the master words of 0, the staging
  // loads of visit -1 and the master words of 1, in that order.
  auto iter = [&](auto firstc, int j, f32x4_t (&w)[4], uint32_t& m, u32x4_t (&sx)[2 * XU],
                  u32x4_t (&sy)[2 * XU]) {
    constexpr bool first = decltype(firstc)::value;
    asm volatile("s_waitcnt vmcnt(%5)"
                 : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]), "+v"(m)
                 : "n"(first ? NX + NW : NX + S + NW)
                 : "memory");
    const int kb = phys(j);
    float wn[16];
    if constexpr (UPD) {
      const uint16_t* xcb = xc + (j & 1) * Ly::cols + l32 * Ly::XC + 8 * lh;
      u32x4_t xa[NBS];
#pragma unroll
      for (int s = 0; s < NBS; ++s) xa[s] = *reinterpret_cast<const u32x4_t*>(xcb + 16 * s);
      f32x16_t d = zero16();
      // one staging load after every second MFMA (NX <= NBS / 2)
#pragma unroll
      for (int s = 0; s < NBS; ++s) {
        d = mma32(xa[s], gs[s], d);
        if ((s & 1) && (s >> 1) < NX) {
          __builtin_amdgcn_sched_barrier(0);
          load_x1(j, s >> 1, sx);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if constexpr (FWD && !first) forward((j - 1) & 1);
      // masked update: a sign-extended mask bit selects the new value or +0
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kl = 8 * (r >> 2) + 4 * lh + (r & 3);
        const uint32_t keep = (uint32_t)(((int)(m << (31 - kl))) >> 31);
        wn[r] = __uint_as_float(__float_as_uint(__fsub_rn(w[r >> 2][r & 3], __fmul_rn(lrv, d[r]))) & keep);
      }
      float* wp = wimg + ((size_t)kb * (Np / 32) + grp) * 1024 + lane * 4;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(wp + 256 * q) = make_float4(wn[4 * q], wn[4 * q + 1], wn[4 * q + 2], wn[4 * q + 3]);
    } else {
#pragma unroll
      for (int i = 0; i < NX; ++i) load_x1(j, i, sx);
      if constexpr (FWD && !first) forward((j - 1) & 1);
#pragma unroll
      for (int r = 0; r < 16; ++r) wn[r] = w[r >> 2][r & 3];
    }
    to_bf16x2(wn, pp);
    load_w(min(j + 2, last), w, m);                    // after the last use of this visit's words
    if (a.Wt) {
      // transposed operand copy for the backward of the layer above: the
      // wave's 32 inputs x 32 units go through its LDS tile [k][n], then out
      // as 16-byte pieces of rows k (eight units each)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        tw[(8 * (r >> 2) + 4 * lh + (r & 3)) * Ly::TR + l32] = (uint16_t)(pp[r >> 1] >> (16 * (r & 1)));
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");   // the other lanes' writes before the reads
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      uint16_t* wt = a.Wt + (size_t)v * Kp * Np + (size_t)(32 * kb) * Np + (size_t)grp * 32 + 8 * (lane & 3);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int kk = 16 * h + (lane >> 2);
        const u32x4_t t = *reinterpret_cast<const u32x4_t*>(tw + kk * Ly::TR + 8 * (lane & 3));
        *reinterpret_cast<u32x4_t*>(wt + (size_t)kk * Np) = t;
      }
    }
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(first ? NX + S + 2 * NW : NX + 2 * S + 2 * NW) : "memory");
#pragma unroll
    for (int q = 0; q < 2 * XU; ++q) asm volatile("" : "+v"(sy[q]));
    if (j < last) store_xc((j + 1) & 1, sy);
    store_xr(j & 1, sy);
    __syncthreads();
  };

  // Prologue: the columns of visit 0 into LDS, then the master words of
  // visit 0, the staging loads of visit -1 (columns of 1, rows of 0) and the
  // master words of visit 1 (past the end the last block is re-read in
  // bounds and never used).
  f32x4_t wA[4], wB[4];
  uint32_t mA = 0u, mB = 0u;
#pragma unroll
  for (int i = 0; i < NX; ++i)
    if (UPD && i < XU) load_x1(-2, i, stE);            // columns of visit 0
  load_w(0, wA, mA);
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(NW) : "memory");
#pragma unroll
  for (int q = 0; q < 2 * XU; ++q) asm volatile("" : "+v"(stE[q]));
  store_xc(0, stE);
  __syncthreads();                                     // (the bias of this lane is read by this lane only)
  if (UPD && lh == 0) a.bias[(size_t)v * Np + n] = bias_n;
#pragma unroll
  for (int i = 0; i < NX; ++i) load_x1(-1, i, stO);   // columns of visit 1, rows of visit 0
  load_w(min(1, last), wB, mB);
  // whole pairs of visits (the block count is even): the register sets keep
  // their roles on every path, so no copy of a set in flight is ever needed
  const std::true_type first{};
  const std::false_type later{};
  iter(first, 0, wA, mA, stE, stO);
  iter(later, 1, wB, mB, stO, stE);
  for (int j = 2; j < nkb; j += 2) {
    iter(later, j, wA, mA, stE, stO);
    iter(later, j + 1, wB, mB, stO, stE);
  }
  if constexpr (FWD) forward(last & 1);
  // the unused prefetches of the last visits land before their registers are reused
  asm volatile("s_waitcnt vmcnt(0)"
               : "+v"(wA[0]), "+v"(wA[1]), "+v"(wA[2]), "+v"(wA[3]), "+v"(mA), "+v"(wB[0]), "+v"(wB[1]),
                 "+v"(wB[2]), "+v"(wB[3]), "+v"(mB)
               :
               : "memory");
#pragma unroll
  for (int q = 0; q < 2 * XU; ++q) asm volatile("" : "+v"(stE[q]), "+v"(stO[q]));

  if constexpr (FWD) {
    // bias, ReLU, bf16 rows [b][n] and columns [n][b]
    uint16_t* orow = a.Orows + a.or_vs * v;
    uint16_t* ocol = a.Ocols ? a.Ocols + a.oc_vs * v : nullptr;
#pragma unroll
    for (int T = 0; T < BT; ++T) {
      float f[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float zz = z[T][r] + bias_n;
        f[r] = zz > 0.0f ? zz : 0.0f;
      }
      uint32_t pk[8];
      to_bf16x2(f, pk);
#pragma unroll
      for (int r = 0; r < 16; ++r)
        orow[(size_t)(32 * T + crow(r, lane)) * Np + n] = (uint16_t)(pk[r >> 1] >> (16 * (r & 1)));
      if (ocol)
#pragma unroll
        for (int q = 0; q < 4; ++q)                    // rows 32T + 8q + 4lh + 0..3 are consecutive
          *reinterpret_cast<u32x2_t*>(ocol + (size_t)n * BP + 32 * T + 8 * q + 4 * lh) = u32x2_t{pk[2 * q], pk[2 * q + 1]};
    }
  }
  vt_add(a.vtime, v, vt0);
}

bool stream_layer_supported(int Kp, int Np, int Bp, int R) {
  return Kp % 64 == 0 && Kp > 0 && Np % kSU == 0 && (Bp == 128 || Bp == 256) && R == Bp;
}

template <int BP, bool UPD, bool FWD>
static hipError_t launch_s(const LayerArgs<uint16_t>& a, int P, hipStream_t s, const LaunchEv& ev) {
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_stream_layer<BP, UPD, FWD>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)StreamLds<BP>::bytes);
    attr = true;
  }
  hipExtLaunchKernelGGL((k_stream_layer<BP, UPD, FWD>), dim3(a.Np / kSU, P), dim3(kST), StreamLds<BP>::bytes, s,
                        ev.start, ev.stop, 0, a);
  return hipGetLastError();
}

template <int BP>
static hipError_t launch_bp(const LayerArgs<uint16_t>& a, int P, hipStream_t s, const LaunchEv& ev) {
  if (a.do_update && a.do_forward) return launch_s<BP, true, true>(a, P, s, ev);
  if (a.do_update) return launch_s<BP, true, false>(a, P, s, ev);
  return launch_s<BP, false, true>(a, P, s, ev);
}

hipError_t launch_stream_layer(const LayerArgs<uint16_t>& a, int P, hipStream_t s, const LaunchEv& ev) {
  if (!a.do_update && !a.do_forward) return hipSuccess;
  if (!stream_layer_supported(a.Kp, a.Np, a.Bp, a.do_forward ? a.R : a.Bp)) return hipErrorInvalidValue;
  return a.Bp == 256 ? launch_bp<256>(a, P, s, ev) : launch_bp<128>(a, P, s, ev);
}

}  // namespace gevo
