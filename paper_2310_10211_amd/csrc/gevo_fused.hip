// Fused per-variant training kernel for two-layer nets (bf16 operands, fp32
// master weights): one persistent workgroup owns one variant for a whole run
// of SGD steps (paper section 6.2 update rule; fitness by retraining, section
// 4.3).  Variants never exchange data, so workgroups are fully independent.
//
// Per step t, for hidden width HP and batch tile BP
// (one wave per 32 hidden units, HP/32 waves):
//   A1 = relu(Z1 + b1) -> LDS (bf16), ReLU' bits kept in registers
//   logits = A1 W2^T + b2, softmax cross-entropy, argmax, G2 = (p - y) / b
//   G1 = (G2 W2) * ReLU'   (old W2),   dW2 = G2^T A1,  W2, b2, b1 updated
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
// over b) feeds dW1 and how the updated W1 (accumulators over k) feeds the
// forward pass without leaving registers.
#include "gevo_internal.h"
#include "gevo_device.h"

#include <hip/hip_ext.h>
#include <math.h>

namespace gevo {

namespace {

__device__ __forceinline__ uint4 ld2x8(const uint16_t* p0, const uint16_t* p1) {
  const uint2 lo = *reinterpret_cast<const uint2*>(p0);
  const uint2 hi = *reinterpret_cast<const uint2*>(p1);
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}

__device__ __forceinline__ uint32_t pack2(uint16_t lo, uint16_t hi) { return (uint32_t)lo | ((uint32_t)hi << 16); }

__device__ __forceinline__ float f4get(const float4& f, int i) {
  return i == 0 ? f.x : (i == 1 ? f.y : (i == 2 ? f.z : f.w));
}

}  // namespace

template <int HP, int BP>
struct Fused2Lds {
  static constexpr int XR = 32 + 8;      // X row block [BP][32]
  static constexpr int XC = BP + 8;      // X col block [32][BP]
  static constexpr int AS = HP + 8;      // A1 [BP][HP]
  static constexpr int W2S = HP + 8;     // W2 operand [32][HP]
  static constexpr int W2T = 32 + 8;     // W2 operand transposed [HP][32]
  static constexpr int GS = 32 + 8;      // G2 [BP][32]
  static constexpr size_t xr = 0;
  static constexpr size_t xc = xr + 2ull * BP * XR * 2;
  static constexpr size_t a1 = xc + 2ull * 32 * XC * 2;
  static constexpr size_t w2 = a1 + (size_t)BP * AS * 2;
  static constexpr size_t w2t = w2 + 32ull * W2S * 2;
  static constexpr size_t g2 = w2t + (size_t)HP * W2T * 2;
  static constexpr size_t b2 = g2 + (size_t)BP * GS * 2;
  static constexpr int NW = HP / 32;    // waves
  static constexpr size_t m2 = b2 + 32 * 4;                  // [32][HP/32] W2 mask words
  static constexpr size_t rce = m2 + 32 * (HP / 32) * 4;     // [BP] per-row loss
  static constexpr size_t rco = rce + (size_t)BP * 8;        // [BP] per-row hit
  static constexpr size_t bytes = rco + (size_t)BP * 4;
  static_assert((size_t)BP * 33 * 4 + (size_t)NW * 2 * 32 * 4 <= a1, "layer-2 staging must fit in the X buffers");
};

template <int HP, int BP>
__global__ __launch_bounds__(2 * HP, 1) void k_fused2(Fused2Args a) {
  using O = Op<uint16_t>;
  typedef uint4 F;
  typedef Fused2Lds<HP, BP> Ly;
  constexpr int NW = Ly::NW;                 // waves, one per 32 hidden units
  constexpr int NT = 64 * NW;                // threads
  constexpr int XU = (4 * BP + NT - 1) / NT; // 16-byte X chunks per thread per block
  constexpr int BT = BP / 32;                // batch tiles
  constexpr int NBS = BP / 16;               // contraction steps over the batch
  constexpr int ZS = 33;                     // row stride of the fp32 logit staging
  extern __shared__ __align__(16) char smem[];
  uint16_t* xr = reinterpret_cast<uint16_t*>(smem + Ly::xr);
  uint16_t* xc = reinterpret_cast<uint16_t*>(smem + Ly::xc);
  uint16_t* a1 = reinterpret_cast<uint16_t*>(smem + Ly::a1);
  uint16_t* w2 = reinterpret_cast<uint16_t*>(smem + Ly::w2);
  uint16_t* w2t = reinterpret_cast<uint16_t*>(smem + Ly::w2t);
  uint16_t* g2 = reinterpret_cast<uint16_t*>(smem + Ly::g2);
  float* b2s = reinterpret_cast<float*>(smem + Ly::b2);
  uint32_t* m2s = reinterpret_cast<uint32_t*>(smem + Ly::m2);
  double* red_row_ce = reinterpret_cast<double*>(smem + Ly::rce);
  unsigned int* red_row_co = reinterpret_cast<unsigned int*>(smem + Ly::rco);
  // layer-2 phase scratch, aliasing the X staging buffers (idle between passes)
  float* zb = reinterpret_cast<float*>(smem + Ly::xr);                    // [BP][ZS]
  float* dbpart = zb + BP * ZS;                                           // [NW][32]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, lh = lane >> 5;
  const int v = blockIdx.x;
  const int Kp = a.Kp, nkb = Kp / 32, kw1 = Kp / 32;
  const int n = wave * 32 + l32;             // hidden unit of this lane's column
  float* W1 = a.W1 + (size_t)v * HP * Kp;
  const uint32_t* m1 = a.m1 + (size_t)v * HP * kw1;
  float* W2 = a.W2 + (size_t)v * 32 * HP;
  const uint32_t* m2 = a.m2 + (size_t)v * 32 * (HP / 32);
  const float lrv = a.lr[v];

  // resident layer 2: fp32 master of this lane's 16 (class, unit) pairs in
  // registers, bf16 operand copies in both orientations and the mask in LDS
  float w2r[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) w2r[r] = W2[((size_t)wave * 32 + crow(r, lane)) * 32 + l32];
  for (int i = tid; i < 32 * HP; i += NT) {      // W2 k-blocked [HP/32][32][32]
    const int c = (i >> 5) & 31, nn = (i >> 10) * 32 + (i & 31);
    const uint16_t u = O::from_f32(W2[i]);
    w2[c * Ly::W2S + nn] = u;
    w2t[nn * Ly::W2T + c] = u;
  }
  if (tid < 32) b2s[tid] = a.b2[(size_t)v * 32 + tid];
  for (int i = tid; i < 32 * (HP / 32); i += NT) m2s[i] = m2[i];
  float b1v = a.b1[(size_t)v * HP + n];
  double ce_tot = 0.0;
  unsigned long long corr_tot = 0;
  if (tid == 0) {
    ce_tot = a.ce_acc[v];
    corr_tot = a.correct_acc[v];
  }

  f32x16_t zacc[BT];
  F g1p[NBS];

  // ---- head of the next pass over the input columns, loaded into registers
  //      ahead of time: X blocks 0 and 1, W1 block 0 and its mask words, and
  //      the labels of the step whose loss the pass prepares
  uint4 xr0[XU], xc0[XU], xr1[XU], xc1[XU];
  float4 wn[4];
  uint32_t mwn = 0;
  int ylab = -1;
  auto load_x = [&](bool upd, int tu, bool fwd, int tf, int kb, uint4 (&xrn)[XU], uint4 (&xcn)[XU]) {
    const uint16_t* xrs = a.xrows + (size_t)tf * BP * Kp;
    const uint16_t* xcs = a.xcols + (size_t)tu * Kp * BP;
#pragma unroll
    for (int u = 0; u < XU; ++u) {
      xrn[u] = xcn[u] = make_uint4(0, 0, 0, 0);
      const int i = tid + NT * u;
      if (kb < nkb && i < 4 * BP) {
        if (fwd) {
          const int b = i >> 2, q = i & 3;
          xrn[u] = *reinterpret_cast<const uint4*>(xrs + (size_t)b * Kp + kb * 32 + q * 8);
        }
        if (upd) {
          const int k = i / (BP / 8), q = i % (BP / 8);
          xcn[u] = *reinterpret_cast<const uint4*>(xcs + (size_t)(kb * 32 + k) * BP + q * 8);
        }
      }
    }
  };
  auto store_x = [&](bool upd, bool fwd, int buf, const uint4 (&xrn)[XU], const uint4 (&xcn)[XU]) {
#pragma unroll
    for (int u = 0; u < XU; ++u) {
      const int i = tid + NT * u;
      if (i < 4 * BP) {
        if (fwd) {
          const int b = i >> 2, q = i & 3;
          *reinterpret_cast<uint4*>(xr + buf * BP * Ly::XR + b * Ly::XR + q * 8) = xrn[u];
        }
        if (upd) {
          const int k = i / (BP / 8), q = i % (BP / 8);
          *reinterpret_cast<uint4*>(xc + buf * 32 * Ly::XC + k * Ly::XC + q * 8) = xcn[u];
        }
      }
    }
  };
  auto issue_head = [&](bool upd, int tu, bool fwd, int tf) {
    load_x(upd, tu, fwd, tf, 0, xr0, xc0);
    load_x(upd, tu, fwd, tf, 1, xr1, xc1);
#pragma unroll
    for (int q = 0; q < 4; ++q) wn[q] = *reinterpret_cast<const float4*>(W1 + (size_t)n * 32 + 8 * q + 4 * lh);
    mwn = upd ? m1[(size_t)n * kw1] : 0u;
    if (fwd && tid < BP) ylab = a.labels[(size_t)tf * BP + tid];
  };

  // ---- one pass over the input columns (head already issued): optional dW1 +
  //      update (step tu), optional forward accumulation of step tf into zacc
  auto kloop = [&](bool upd, int tu, bool fwd, int tf) {
    if (fwd) {
#pragma unroll
      for (int T = 0; T < BT; ++T) zacc[T] = zero16();
    }
    store_x(upd, fwd, 0, xr0, xc0);
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
      const int buf = kb & 1;
      const bool more = kb + 1 < nkb;
      uint4 xr2[XU], xc2[XU];
      load_x(upd, tu, fwd, tf, kb + 2, xr2, xc2);
      float4 wc[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) wc[q] = wn[q];
      const uint32_t mw = mwn;
      if (more) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          wn[q] = *reinterpret_cast<const float4*>(W1 + ((size_t)(kb + 1) * HP + n) * 32 + 8 * q + 4 * lh);
        mwn = upd ? m1[(size_t)n * kw1 + kb + 1] : 0u;
      }
      const uint16_t* xcb = xc + buf * 32 * Ly::XC;
      const uint16_t* xrb = xr + buf * BP * Ly::XR;
      float wnew[16];
      if (upd) {
        f32x16_t dacc = zero16();
#pragma unroll
        for (int s = 0; s < NBS; ++s) {
          const uint16_t* pp = xcb + l32 * Ly::XC + 16 * s + 4 * lh;
          dacc = O::mma(ld2x8(pp, pp + 8), g1p[s], dacc);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kl = 8 * (r >> 2) + 4 * lh + (r & 3);
          const bool keep = (mw >> kl) & 1u;
          wnew[r] = keep ? __fsub_rn(f4get(wc[r >> 2], r & 3), __fmul_rn(lrv, dacc[r])) : 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<float4*>(W1 + ((size_t)kb * HP + n) * 32 + 8 * q + 4 * lh) =
              make_float4(wnew[4 * q], wnew[4 * q + 1], wnew[4 * q + 2], wnew[4 * q + 3]);
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) wnew[r] = f4get(wc[r >> 2], r & 3);
      }
      if (fwd) {
        F wb[2];
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const float* q = &wnew[8 * s2];
          wb[s2] = make_uint4(pack2(O::from_f32(q[0]), O::from_f32(q[1])), pack2(O::from_f32(q[2]), O::from_f32(q[3])),
                              pack2(O::from_f32(q[4]), O::from_f32(q[5])), pack2(O::from_f32(q[6]), O::from_f32(q[7])));
        }
#pragma unroll
        for (int T = 0; T < BT; ++T)
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2) {
            const uint16_t* pp = xrb + (32 * T + l32) * Ly::XR + 16 * s2 + 4 * lh;
            zacc[T] = O::mma(ld2x8(pp, pp + 8), wb[s2], zacc[T]);
          }
      }
      if (more) store_x(upd, fwd, buf ^ 1, xr1, xc1);
#pragma unroll
      for (int u = 0; u < XU; ++u) { xr1[u] = xr2[u]; xc1[u] = xc2[u]; }
      __syncthreads();
    }
  };

  // prologue: forward of the first step
  issue_head(false, 0, true, a.t0);
  kloop(false, 0, true, a.t0);

  for (int t = a.t0; t < a.t1; ++t) {
    const int64_t r0 = (int64_t)t * a.B;
    const int bt = (int)((a.n - r0) < a.B ? (a.n - r0) : a.B);
    const float scale = __fdiv_rn(1.0f, (float)bt);
    // ---- A1 = relu(Z1 + b1) -> LDS, ReLU' bits
    uint32_t rb[BT];
#pragma unroll
    for (int T = 0; T < BT; ++T) {
      uint32_t bits = 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float z = zacc[T][r] + b1v;
        const uint16_t u = O::from_f32(z > 0.0f ? z : 0.0f);
        a1[(32 * T + crow(r, lane)) * Ly::AS + n] = u;
        bits |= (uint32_t)(u != 0) << r;
      }
      rb[T] = bits;
    }
    __syncthreads();
    // ---- logits (MFMA, one batch tile per wave) -> LDS
    if (wave < BT) {
      f32x16_t c0 = zero16(), c1 = zero16();
      const uint16_t* ap = a1 + (32 * wave + l32) * Ly::AS + 8 * lh;
      const uint16_t* bp = w2 + l32 * Ly::W2S + 8 * lh;
#pragma unroll
      for (int s = 0; s < HP / 16; s += 2) {
        c0 = O::mma(O::load(ap + 16 * s), O::load(bp + 16 * s), c0);
        c1 = O::mma(O::load(ap + 16 * s + 16), O::load(bp + 16 * s + 16), c1);
      }
      const float bias_c = b2s[l32];
#pragma unroll
      for (int r = 0; r < 16; ++r) zb[(32 * wave + crow(r, lane)) * ZS + l32] = (c0[r] + c1[r]) + bias_c;
    }
    __syncthreads();
    // ---- per row (one thread each): softmax cross-entropy, argmax (lowest index
    //      on ties, a NaN logit is a miss), G2 = (p - onehot(y)) * fl(1/b)
    if (tid < BP) {
      const int b = tid, C = a.C, y = ylab;
      float* zr = zb + b * ZS;
      float m = zr[0], bv = zr[0];
      int bi = 0, isn = zr[0] != zr[0];
      for (int c = 1; c < C; ++c) {
        const float z = zr[c];
        if (z != z) isn = 1;
        else if (z > bv) { bv = z; bi = c; }
        m = fmaxf(m, z);
      }
      float s = 0.0f;
      for (int c = 0; c < C; ++c) s += expf(zr[c] - m);
      const bool rvalid = y >= 0;
      float ce = (logf(s) + m) - zr[rvalid ? y : 0];
      if (isn) ce = NAN;
      red_row_ce[b] = rvalid ? (double)ce : 0.0;
      red_row_co[b] = (rvalid && !isn && bi == y) ? 1u : 0u;
      for (int c = 0; c < 32; ++c) {
        float g = 0.0f;
        if (c < C && rvalid) g = (expf(zr[c] - m) / s - (c == y ? 1.0f : 0.0f)) * scale;
        zr[c] = g;                                                // fp32 gradient for db2
        g2[b * Ly::GS + c] = O::from_f32(g);
      }
    }
    __syncthreads();
    // ---- reductions in a fixed order: db2 partials over row groups, loss and hits
    {
      const int c = tid & 31, part = tid >> 5;                    // NW*2 parts of rows
      float sp = 0.0f;
      for (int b = part; b < BP; b += 2 * NW) sp += zb[b * ZS + c];
      dbpart[part * 32 + c] = sp;
    }
    if (wave == 0) {
      double sc = 0.0;
      unsigned int co = 0;
      for (int b = lane; b < BP; b += 64) { sc += red_row_ce[b]; co += red_row_co[b]; }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) { sc += __shfl_xor(sc, off); co += __shfl_xor(co, off); }
      if (lane == 0) { ce_tot += sc; corr_tot += co; }
    }
    __syncthreads();
    if (tid < 32) {
      float db = 0.0f;
#pragma unroll
      for (int part = 0; part < 2 * NW; ++part) db += dbpart[part * 32 + tid];
      b2s[tid] = __fsub_rn(b2s[tid], __fmul_rn(lrv, db));      // read again only next step
    }
    // ---- G1 = (G2 W2) * ReLU' with the pre-update W2 (accumulators reuse zacc)
#pragma unroll
    for (int T = 0; T < BT; ++T) {
      f32x16_t acc = zero16();
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
        acc = O::mma(O::load(g2 + (32 * T + l32) * Ly::GS + 16 * s2 + 8 * lh),
                     O::load(w2t + n * Ly::W2T + 16 * s2 + 8 * lh), acc);
      zacc[T] = acc;
    }
    float db1p = 0.0f;
#pragma unroll
    for (int T = 0; T < BT; ++T) {
      uint16_t u[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        u[r] = O::from_f32(((rb[T] >> r) & 1u) ? zacc[T][r] : 0.0f);
        db1p += O::to_f32(u[r]);
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
        g1p[2 * T + s2] = make_uint4(pack2(u[8 * s2], u[8 * s2 + 1]), pack2(u[8 * s2 + 2], u[8 * s2 + 3]),
                                     pack2(u[8 * s2 + 4], u[8 * s2 + 5]), pack2(u[8 * s2 + 6], u[8 * s2 + 7]));
    }
    db1p += __shfl_xor(db1p, 32);
    b1v = __fsub_rn(b1v, __fmul_rn(lrv, db1p));
    // the next pass's first blocks, W1 words and labels can load from here on
    const bool fwd_next = t + 1 < a.t1;
    issue_head(true, t, fwd_next, t + 1);
    // ---- dW2 = G2^T A1 (classes x hidden), reads of LDS only
    f32x16_t d2 = zero16();
#pragma unroll
    for (int s = 0; s < NBS; ++s)
      d2 = O::mma(O::gather(g2 + (16 * s + 8 * lh) * Ly::GS + l32, Ly::GS),
                  O::gather(a1 + (16 * s + 8 * lh) * Ly::AS + n, Ly::AS), d2);
    __syncthreads();
    // ---- masked SGD on W2 (register master) and refresh of its LDS operands
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int c = crow(r, lane);
      const bool keep = (m2s[c * (HP / 32) + (n >> 5)] >> (n & 31)) & 1u;
      w2r[r] = keep ? __fsub_rn(w2r[r], __fmul_rn(lrv, d2[r])) : 0.0f;
      const uint16_t u = O::from_f32(w2r[r]);
      w2[c * Ly::W2S + n] = u;
      w2t[n * Ly::W2T + c] = u;
    }
    // ---- dW1 + masked SGD on W1 + forward of the next step
    kloop(true, t, fwd_next, t + 1);
  }
  // ---- write back the resident state
#pragma unroll
  for (int r = 0; r < 16; ++r) W2[((size_t)wave * 32 + crow(r, lane)) * 32 + l32] = w2r[r];
  if (lh == 0) a.b1[(size_t)v * HP + n] = b1v;
  if (tid < 32) a.b2[(size_t)v * 32 + tid] = b2s[tid];
  if (tid == 0) {
    a.ce_acc[v] = ce_tot;
    a.correct_acc[v] = corr_tot;
  }
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
