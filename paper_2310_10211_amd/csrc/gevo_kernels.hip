// HIP kernels of libgevo for CDNA4 (gfx950): population-batched training and
// prediction of small fully-connected classifiers (fitness evaluation of
// GEVO-ML, arXiv 2310.10211, section 4.3; SGD update of section 6.2).
//
// Device layout (per variant v, layer l with padded input width Kp and padded
// output width Np, both multiples of 32):
//   Wm   fp32 master weights, k-blocked [v][Kp/32][Np][32]: element (n, k) at
//        ((k/32)*Np + n)*32 + k%32, so every 32-column block is one contiguous run
//   bias fp32 [v][Np]
//   mask uint32 row words, [v][Np][Kp/32] (bit k%32 of word [n][k/32])
// Activations and gradients come in two orientations: "rows" [v][b][feature]
// (feature contiguous) and "cols" [v][feature][b] (batch contiguous), so that
// every MFMA operand is read along its contraction index.
//
// GEMMs run on v_mfma_f32_32x32x16_bf16 (bf16 path) or v_mfma_f32_32x32x2_f32
// (fp32 path).  Fragment layout of a 32x32xK MFMA with E elements per lane
// (E = 8 for bf16, 1 for fp32): lane l supplies A[l%32][(l/32)*E + i] and
// B[(l/32)*E + i][l%32]; the 16 accumulators of lane l hold
// C[8*(r/4) + 4*(l/32) + r%4][l%32], r = 0..15.
#include "gevo_internal.h"
#include "gevo_device.h"

#include <hip/hip_ext.h>
#include <math.h>

namespace gevo {

// ------------------------------------------------------------ population init
// One thread per (variant, padded output row n, 32-wide word of inputs k):
// draws the 32 mask bits and initial weights of W_l[n][k0..k0+31].  Rows n
// are the fastest index, so a wave writes one contiguous 8 KiB span of the
// k-blocked master, four weights per store.
// The base-noise draw eps = sqrt(-2 ln u1) cos(2 pi u2) uses the hardware
// log2 and cos(2 pi x) instructions: their error moves eps by about 1e-6
// relative, i.e. the weight w (1 + 0.01 eps) by about 1e-8.
__global__ __launch_bounds__(256) void k_init(InitArgs a) {
  const int words = a.Kp / 32;
  const int64_t total = (int64_t)a.P * a.Np * words;
  const uint2 key = make_uint2((uint32_t)(a.seed & 0xffffffffu), (uint32_t)(a.seed >> 32));
  const float two_m24 = 5.9604644775390625e-08f;   // 2^-24
  for (int64_t it = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; it < total;
       it += (int64_t)gridDim.x * blockDim.x) {
    const int n = (int)(it % a.Np);
    const int kw = (int)((it / a.Np) % words);
    const int v = (int)(it / ((int64_t)words * a.Np));
    uint32_t bits = 0;
    if (a.ident && a.ident[v]) {                   // a removed layer: its identity form
      const int win = (int)a.width_in[v], wout = (int)a.width_out[v], m = win < wout ? win : wout;
      float* wrow = a.Wm + (size_t)v * a.Np * a.Kp + ((size_t)kw * a.Np + n) * 32;
      for (int q = 0; q < 8; ++q) {
        float wq[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int j = 4 * q + jj, k = kw * 32 + j;
          const bool one = k == n && n < m;
          wq[jj] = one ? 1.0f : 0.0f;
          bits |= (uint32_t)one << j;
        }
        *reinterpret_cast<float4*>(wrow + 4 * q) = make_float4(wq[0], wq[1], wq[2], wq[3]);
      }
      if (kw == 0) a.bias[(size_t)v * a.Np + n] = (n >= win && n < wout) ? 1.0f : 0.0f;
    } else {
      const uint32_t th = a.thresh[v];
      float* wrow = a.Wm + (size_t)v * a.Np * a.Kp + ((size_t)kw * a.Np + n) * 32;
      uint64_t blk_m = ~0ull, blk_i = ~0ull, blk_n = ~0ull;
      uint4 rm = make_uint4(0, 0, 0, 0), ri = rm, rn = rm;
      const bool kept_row = !a.width_out || n < (int)a.width_out[v];
      for (int q = 0; q < 8; ++q) {
        float wq[4];
        float4 bq = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (a.base_w && n < a.N) bq = *reinterpret_cast<const float4*>(a.base_w + (size_t)n * a.Kp + kw * 32 + 4 * q);
        const float bqa[4] = {bq.x, bq.y, bq.z, bq.w};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int j = 4 * q + jj, k = kw * 32 + j;
          float w = 0.0f;
          const bool kept_unit = kept_row && (!a.width_out || k < (int)a.width_in[v]);
          if (n < a.N && k < a.K) {
            const uint64_t e = (uint64_t)n * (uint64_t)a.K + (uint64_t)k;
            bool keep;
            if (a.prune_off) {
              keep = true;
              for (uint32_t pq = a.prune_off[v]; pq < a.prune_off[v + 1]; ++pq) {
                const uint4 r = philox(make_uint4((uint32_t)(e >> 2), (uint32_t)a.l_index, a.prune_id[pq], kStreamMask), key);
                if ((pick(r, (uint32_t)(e & 3)) >> 8) >= a.prune_th[pq]) keep = false;
              }
            } else {
              if ((e >> 2) != blk_m) {
                blk_m = e >> 2;
                rm = philox(make_uint4((uint32_t)blk_m, (uint32_t)a.l_index, (uint32_t)v, kStreamMask), key);
              }
              keep = (pick(rm, (uint32_t)(e & 3)) >> 8) < th;
            }
            if (a.base_w) {
              w = bqa[jj];
            } else {
              if ((e >> 2) != blk_i) {
                blk_i = e >> 2;
                ri = philox(make_uint4((uint32_t)blk_i, (uint32_t)a.l_index, 0u, kStreamInit), key);
              }
              const float u = (float)(pick(ri, (uint32_t)(e & 3)) >> 8) * two_m24;
              const float t = __fsub_rn(__fmul_rn(2.0f, u), 1.0f);       // exact
              w = __fmul_rn(t, a.xavier_a);
            }
            if (a.init_kind == 1) {
              if ((e >> 1) != blk_n) {
                blk_n = e >> 1;
                rn = philox(make_uint4((uint32_t)blk_n, (uint32_t)a.l_index, (uint32_t)v, kStreamNoise), key);
              }
              const uint32_t w0 = (uint32_t)(e & 1) * 2u;
              const float u1 = (float)((pick(rn, w0) >> 8) + 1u) * two_m24;   // (0, 1]
              const float u2 = (float)(pick(rn, w0 + 1) >> 8) * two_m24;      // [0, 1)
              // -2 ln u1 = -2 ln(2) log2(u1); cos(2 pi u2) takes u2 in turns
              const float eps = __builtin_amdgcn_sqrtf(-1.3862943611198906f * __builtin_amdgcn_logf(u1)) *
                                __builtin_amdgcn_cosf(u2);
              w = __fmul_rn(w, __fadd_rn(1.0f, __fmul_rn(a.noise_std, eps)));
            }
            keep = keep && kept_unit;
            if (!keep) w = 0.0f;
            bits |= (uint32_t)keep << j;
          }
          wq[jj] = w;
        }
        *reinterpret_cast<float4*>(wrow + 4 * q) = make_float4(wq[0], wq[1], wq[2], wq[3]);
      }
      if (kw == 0) {
        const bool bk = n < a.N && (!a.width_out || (n < (int)a.width_out[v] && a.bias_keep[v]));
        a.bias[(size_t)v * a.Np + n] = (a.base_b && bk) ? a.base_b[n] : 0.0f;
      }
    }
    a.mask[((size_t)v * a.Np + n) * words + kw] = bits;
  }
}

// ------------------------------------------------------------ hidden layer
// Workgroup (n-tile of 32 output units, variant v); four waves.  The inputs
// k are processed in blocks of KB columns (the block's operand copy of W fits
// in LDS).  Update (do_update), per 32-wide chunk c of a block, each wave
// streaming its own chunks with the next chunk's weights already in flight:
//   dW^T[n][k] = sum_b G[n][b] * A[k][b]          (MFMA, contraction = batch)
// staged through LDS, then lane (row n, 16 columns) applies
//   W[n][k]    = mask ? fl(W - fl(lr * dW)) : +0   (fp32 master, float4 in place)
// and b[n] -= lr * sum_b G[n][b].  The updated block stays in LDS as an
// operand, so the forward pass of the next step runs without re-reading W:
//   Z[r][n] = sum_k A_next[r][k] * W[n][k] + b[n],  A_out = relu(Z)  (MFMA)
// Without do_update a block is loaded from the master (forward only).
template <typename S, int BPMAX>
__global__ __launch_bounds__(256, 2) void k_layer(LayerArgs<S> a) {
  using O = Op<S>;
  using F = typename O::Frag;
  constexpr int KM = O::KM, KE = O::KE;
  constexpr int NG = BPMAX / KM;
  constexpr int TPW = BPMAX / 128;                   // row tiles per wave in a forward pass
  constexpr int PASS = BPMAX;                        // rows per forward pass
  constexpr int DSTR = 36;                           // fp32 staging row stride (16-byte aligned rows)
  constexpr int SSTR = 32 + O::PAD;
  extern __shared__ __align__(16) char smem[];
  __shared__ float bias_l[32];
  const int KB = a.KB, WS = KB + O::PAD;
  S* wt = reinterpret_cast<S*>(smem);                                // [32][WS] operand tile
  float* stage = reinterpret_cast<float*>(smem + (size_t)32 * WS * sizeof(S));   // [4][32][DSTR]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, lh = lane >> 5;
  const int n0 = blockIdx.x * 32, v = blockIdx.y;
  const uint64_t vt0 = vt_now();
  if (a.wout && n0 >= (int)a.wout[v]) {                  // every unit of the tile removed
    vt_add(a.vtime, v, vt0);
    return;
  }
  const int Kp = a.Kp, Np = a.Np, kwords = Kp / 32;
  float* Wv = a.Wm + (size_t)v * Np * Kp;                     // this variant, k-blocked
  const uint32_t* mk = a.mask + ((size_t)v * Np + n0) * kwords;
  const float lrv = a.lr[v];
  const int nsteps = a.Bp / KM;
  float* dws = stage + wave * 32 * DSTR;
  const int rn = lane >> 1, cs = (lane & 1) * 16;            // update ownership: row rn, columns cs..cs+15

  F gf[NG];
  if (a.do_update) {
    const S* G = a.Gcols + v * a.g_vs;
    // the gradient operand of dW first, so its loads are in flight with the
    // bias gradient's (the bias store below would otherwise hold them back)
    if constexpr (sizeof(S) == 4) {
      // fp32: contraction step s2 pairs batch rows s2 (lanes 0-31) and
      // Bp/2 + s2 (lanes 32-63), so a lane's operands are contiguous
      const S* gp = G + (size_t)(n0 + l32) * a.Bp + lh * (a.Bp / 2);
#pragma unroll
      for (int s2 = 0; s2 < NG; ++s2) gf[s2] = s2 < nsteps ? gp[s2] : F{};
    } else {
      const S* gp = G + (size_t)(n0 + l32) * a.Bp + lh * KE;
#pragma unroll
      for (int s2 = 0; s2 < NG; ++s2) gf[s2] = s2 < nsteps ? O::load(gp + s2 * KM) : F{};
    }
    // bias gradient of the 32 units: 8 lanes per unit, fixed-order reduction
    const int nl = threadIdx.x >> 3, seg = threadIdx.x & 7, per = a.Bp / 8;
    const S* gr = G + (size_t)(n0 + nl) * a.Bp + seg * per;
    float s = 0.0f;
    for (int b = 0; b < per; ++b) s += O::to_f32(gr[b]);
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    if (seg == 0) {
      const float bo = a.bias[(size_t)v * Np + n0 + nl];
      const bool bk = (a.bmask[(size_t)v * (Np / 32) + blockIdx.x] >> nl) & 1u;   // n0 = 32 blockIdx.x
      const float bn = bk ? __fsub_rn(bo, __fmul_rn(lrv, s)) : 0.0f;
      a.bias[(size_t)v * Np + n0 + nl] = bn;
      bias_l[nl] = bn;
    }
  } else if (threadIdx.x < 32) {
    bias_l[threadIdx.x] = a.bias[(size_t)v * Np + n0 + threadIdx.x];
  }

  const int nblk = (Kp + KB - 1) / KB;
  const int R = a.do_forward ? a.R : 0;
  const int npass = a.do_forward ? (R + PASS - 1) / PASS : 0;

  // ---- fill the LDS operand tile with block blk (update or plain load), plus Wt
  auto fill = [&](int blk, bool upd) {
    const int kb0 = blk * KB;
    const int kw = min(KB, Kp - kb0);
    const int nchb = kw / 32;
    if (upd) {
      // row rn of the tile in 32-column chunk c of this block
      auto wptr = [&](int c) { return Wv + ((size_t)(kb0 / 32 + c) * Np + n0 + rn) * 32 + cs; };
      const uint32_t* mrow = mk + (size_t)rn * kwords + kb0 / 32;
      const S* acb = a.Acols + v * a.ac_vs + (size_t)(kb0 + l32) * a.Bp + lh * KE;
      float4 nx[4];
      uint32_t nmw = 0;
      if (wave < nchb) {
#pragma unroll
        for (int u = 0; u < 4; ++u) nx[u] = *reinterpret_cast<const float4*>(wptr(wave) + 4 * u);
        nmw = mrow[wave];
      }
      for (int c = wave; c < nchb; c += 4) {
        float4 w4[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) w4[u] = nx[u];
        const uint32_t mw = nmw;
        if (c + 4 < nchb) {
#pragma unroll
          for (int u = 0; u < 4; ++u) nx[u] = *reinterpret_cast<const float4*>(wptr(c + 4) + 4 * u);
          nmw = mrow[c + 4];
        }
        f32x16_t d0 = zero16(), d1 = zero16();
        if constexpr (sizeof(S) == 4) {
          // batch rows s2 and Bp/2 + s2 as above: four steps per 16-byte load
          const float* ap = a.Acols + v * a.ac_vs + (size_t)(kb0 + c * 32 + l32) * a.Bp + lh * (a.Bp / 2);
#pragma unroll
          for (int s4 = 0; s4 < NG; s4 += 4)
            if (s4 < nsteps) {
              const float4 x = *reinterpret_cast<const float4*>(ap + s4);
              d0 = O::mma(gf[s4], x.x, d0);
              d1 = O::mma(gf[s4 + 1], x.y, d1);
              d0 = O::mma(gf[s4 + 2], x.z, d0);
              d1 = O::mma(gf[s4 + 3], x.w, d1);
              if ((s4 & 15) == 12) __builtin_amdgcn_sched_barrier(0);   // at most four loads ahead
            }
        } else {
          const S* ap = acb + (size_t)c * 32 * a.Bp;
#pragma unroll
          for (int s2 = 0; s2 < NG; s2 += 2) {
            if (s2 < nsteps) d0 = O::mma(gf[s2], O::load(ap + s2 * KM), d0);
            if (s2 + 1 < nsteps) d1 = O::mma(gf[s2 + 1], O::load(ap + (s2 + 1) * KM), d1);
          }
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) dws[crow(r, lane) * DSTR + l32] = d0[r] + d1[r];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        float dw[16];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float4 t = *reinterpret_cast<const float4*>(dws + rn * DSTR + cs + 4 * u);
          dw[4 * u] = t.x; dw[4 * u + 1] = t.y; dw[4 * u + 2] = t.z; dw[4 * u + 3] = t.w;
        }
        float wn[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float w = (i & 3) == 0 ? w4[i >> 2].x : (i & 3) == 1 ? w4[i >> 2].y : (i & 3) == 2 ? w4[i >> 2].z : w4[i >> 2].w;
          const bool keep = (mw >> (cs + i)) & 1u;
          wn[i] = keep ? __fsub_rn(w, __fmul_rn(lrv, dw[i])) : 0.0f;
        }
        float* wdst = wptr(c);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          *reinterpret_cast<float4*>(wdst + 4 * u) = make_float4(wn[4 * u], wn[4 * u + 1], wn[4 * u + 2], wn[4 * u + 3]);
        S* od = wt + rn * WS + c * 32 + cs;
#pragma unroll
        for (int i = 0; i < 16; ++i) od[i] = O::from_f32(wn[i]);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      }
    } else {
      const int q = kw / 4;                               // float4 per row
      for (int i = threadIdx.x; i < 32 * q; i += 256 * 4) {
        float4 w4[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int j = i + u * 256;
          // j in memory order: chunk j/256, row (j/8)%32, float4 j%8
          w4[u] = j < 32 * q ? *reinterpret_cast<const float4*>(
                                   Wv + ((size_t)(kb0 / 32 + j / 256) * Np + n0 + (j / 8) % 32) * 32 + (j % 8) * 4)
                             : make_float4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int j = i + u * 256;
          if (j < 32 * q) {
            S* dst = wt + ((j / 8) % 32) * WS + (j / 256) * 32 + (j % 8) * 4;
            dst[0] = O::from_f32(w4[u].x); dst[1] = O::from_f32(w4[u].y);
            dst[2] = O::from_f32(w4[u].z); dst[3] = O::from_f32(w4[u].w);
          }
        }
      }
    }
    __syncthreads();
    if (a.Wt) {
      // transposed operand copy [k][n] for the backward of the layer above
      for (int k = threadIdx.x >> 1; k < kw; k += 128) {
        const int half = threadIdx.x & 1;
        S* dst = a.Wt + (size_t)v * Kp * Np + (size_t)(kb0 + k) * Np + n0 + half * 16;
#pragma unroll
        for (int i = 0; i < 16; ++i) dst[i] = wt[(half * 16 + i) * WS + k];
      }
    }
  };

  // ---- forward over block blk for rows [row0, row0 + 32*ntiles); two accumulator chains per tile
  auto forward = [&](int blk, int row0, int ntiles, f32x16_t (&acc)[TPW][2]) {
    const int kb0 = blk * KB;
    const int kw = min(KB, Kp - kb0);
#pragma unroll
    for (int ti = 0; ti < TPW; ++ti) {
      const int tile = wave + 4 * ti;
      if (tile >= ntiles) continue;
      const S* ar = a.Arows + v * a.ar_vs + (size_t)(row0 + tile * 32 + l32) * Kp + kb0 + lh * KE;
      const S* br = wt + l32 * WS + lh * KE;
      int k = 0;
      if constexpr (sizeof(S) == 4) {
        // fp32: within each 16 inputs, step u pairs inputs u (lanes 0-31) and
        // 8 + u (lanes 32-63), so a lane's row operands are two 16-byte loads
        const float* ar8 = a.Arows + v * a.ar_vs + (size_t)(row0 + tile * 32 + l32) * Kp + kb0 + 8 * lh;
        const float* br8 = wt + l32 * WS + 8 * lh;
        for (; k + 16 <= kw; k += 16) {
          const float4 x0 = *reinterpret_cast<const float4*>(ar8 + k);
          const float4 x1 = *reinterpret_cast<const float4*>(ar8 + k + 4);
          const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
          for (int u = 0; u < 8; u += 2) {
            acc[ti][0] = O::mma(xs[u], br8[k + u], acc[ti][0]);
            acc[ti][1] = O::mma(xs[u + 1], br8[k + u + 1], acc[ti][1]);
          }
        }
      }
      for (; k + 4 * KM <= kw; k += 4 * KM) {
        F x[4], w[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) { x[u] = O::load(ar + k + u * KM); w[u] = O::load(br + k + u * KM); }
        acc[ti][0] = O::mma(x[0], w[0], acc[ti][0]);
        acc[ti][1] = O::mma(x[1], w[1], acc[ti][1]);
        acc[ti][0] = O::mma(x[2], w[2], acc[ti][0]);
        acc[ti][1] = O::mma(x[3], w[3], acc[ti][1]);
      }
      for (; k < kw; k += KM) acc[ti][0] = O::mma(O::load(ar + k), O::load(br + k), acc[ti][0]);
    }
  };

  // ---- epilogue: bias + ReLU, rows store, transposed store staged in LDS
  auto epilogue = [&](int row0, int ntiles, f32x16_t (&acc)[TPW][2]) {
    S* sw = reinterpret_cast<S*>(dws);                      // [32][SSTR] per wave
#pragma unroll
    for (int ti = 0; ti < TPW; ++ti) {
      const int tile = wave + 4 * ti;
      if (tile < ntiles) {                                  // wave-uniform
        const float bn = bias_l[l32];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = crow(r, lane);
          const float z = (acc[ti][0][r] + acc[ti][1][r]) + bn;
          const S sv = O::from_f32(z > 0.0f ? z : 0.0f);
          a.Orows[v * a.or_vs + (size_t)(row0 + tile * 32 + rl) * Np + n0 + l32] = sv;
          sw[l32 * SSTR + rl] = sv;                        // [n][row]
        }
        if (a.Ocols) {
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
          const int nl = lane >> 1, half = lane & 1;
          S* dst = a.Ocols + v * a.oc_vs + (size_t)(n0 + nl) * R + row0 + tile * 32 + half * 16;
#pragma unroll
          for (int i = 0; i < 16; ++i) dst[i] = sw[nl * SSTR + half * 16 + i];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      }
    }
  };

  if (nblk == 1) {
    fill(0, a.do_update != 0);
    __syncthreads();
    for (int pass = 0; pass < npass; ++pass) {
      const int row0 = pass * PASS;
      const int ntiles = min(PASS, R - row0) / 32;
      f32x16_t acc[TPW][2];
#pragma unroll
      for (int ti = 0; ti < TPW; ++ti) { acc[ti][0] = zero16(); acc[ti][1] = zero16(); }
      forward(0, row0, ntiles, acc);
      epilogue(row0, ntiles, acc);
    }
  } else if (npass == 0) {
    for (int blk = 0; blk < nblk; ++blk) {
      fill(blk, a.do_update != 0);
      __syncthreads();
    }
  } else {
    for (int pass = 0; pass < npass; ++pass) {
      const int row0 = pass * PASS;
      const int ntiles = min(PASS, R - row0) / 32;
      f32x16_t acc[TPW][2];
#pragma unroll
      for (int ti = 0; ti < TPW; ++ti) { acc[ti][0] = zero16(); acc[ti][1] = zero16(); }
      for (int blk = 0; blk < nblk; ++blk) {
        fill(blk, a.do_update != 0 && pass == 0);
        __syncthreads();
        forward(blk, row0, ntiles, acc);
        __syncthreads();
      }
      epilogue(row0, ntiles, acc);
    }
  }
  vt_add(a.vtime, v, vt0);
}

// ------------------------------------------------------------ output layer
// Prediction: workgroup = (256-row chunk, variant).  Logits on MFMA (classes
// padded to 32), then per row (32 lanes hold the 32 classes of a row): max,
// NaN flag, sum of exp, log-sum-exp, CE = lse - z_y, and the argmax with the
// lowest index on ties (a NaN logit makes the row a miss); the chunk's CE
// and hit sums go to per-chunk partials.  (Training runs in the two passes
// below.)
constexpr int kOutWaves = 8;

template <typename S>
__global__ __launch_bounds__(64 * kOutWaves) void k_out(OutArgs<S> a) {
  using O = Op<S>;
  using F = typename O::Frag;
  constexpr int KM = O::KM, KE = O::KE;
  constexpr int NW = kOutWaves;
  constexpr int NT = 64 * NW;
  extern __shared__ __align__(16) char smem[];
  __shared__ double red_ce[NW];
  __shared__ unsigned int red_corr[NW];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, lh = lane >> 5;
  const int v = blockIdx.y, chunk = blockIdx.x;
  const uint64_t vt0 = vt_now();
  const int Kp = a.Kp, WS = Kp + O::PAD;
  S* wop = reinterpret_cast<S*>(smem);                  // [32][WS]  W_L as operand, [class][k]
  const float* Wm = a.Wm + (size_t)v * 32 * Kp;
  {
    const int q = Kp / 4;                                // float4 per row
    for (int i = threadIdx.x; i < 32 * q; i += NT * 4) {
      float4 w4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = i + u * NT;
        w4[u] = j < 32 * q ? *reinterpret_cast<const float4*>(Wm + (size_t)j * 4) : make_float4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = i + u * NT;
        if (j < 32 * q) {
          S* dst = wop + ((j / 8) % 32) * WS + (j / 256) * 32 + (j % 8) * 4;   // row (j/8)%32, chunk j/256
          dst[0] = O::from_f32(w4[u].x); dst[1] = O::from_f32(w4[u].y);
          dst[2] = O::from_f32(w4[u].z); dst[3] = O::from_f32(w4[u].w);
        }
      }
    }
  }
  const float bias_c = a.bias[(size_t)v * 32 + l32];
  __syncthreads();

  const int row_base = chunk * kOutRows;
  const int rows = min(kOutRows, a.rows - row_base);
  const int ntiles = rows / 32;
  const bool cvalid = l32 < a.C;
  double ce_sum = 0.0;
  unsigned int corr = 0;
  for (int tile = wave; tile < ntiles; tile += NW) {
    f32x16_t acc0 = zero16(), acc1 = zero16();
    const S* ar = a.Arows + v * a.ar_vs + (size_t)(row_base + tile * 32 + l32) * Kp + lh * KE;
    const S* wr = wop + l32 * WS + lh * KE;
    int k = 0;
    for (; k + 4 * KM <= Kp; k += 4 * KM) {
      F x[4], w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) { x[u] = O::load(ar + k + u * KM); w[u] = O::load(wr + k + u * KM); }
      acc0 = O::mma(x[0], w[0], acc0);
      acc1 = O::mma(x[1], w[1], acc1);
      acc0 = O::mma(x[2], w[2], acc0);
      acc1 = O::mma(x[3], w[3], acc1);
    }
    for (; k < Kp; k += KM) acc0 = O::mma(O::load(ar + k), O::load(wr + k), acc0);
    int ylab[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) ylab[r] = a.labels[row_base + tile * 32 + crow(r, lane)];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int y = ylab[r];
      const float z = (acc0[r] + acc1[r]) + bias_c;
      int isn = (cvalid && (z != z)) ? 1 : 0;
      float m = cvalid ? z : -INFINITY;
      float bv = (cvalid && !isn) ? z : -INFINITY;
      int bi = l32;
#pragma unroll
      for (int off = 16; off >= 1; off >>= 1) {
        m = fmaxf(m, __shfl_xor(m, off));
        isn |= __shfl_xor(isn, off);
        const float ov = __shfl_xor(bv, off);
        const int oi = __shfl_xor(bi, off);
        if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
      }
      const float e = cvalid ? expf(z - m) : 0.0f;
      float s = e;
#pragma unroll
      for (int off = 16; off >= 1; off >>= 1) s += __shfl_xor(s, off);
      const float zy = __shfl(z, (lane & 32) | (y & 31));
      const bool rvalid = y >= 0;
      float ce = (logf(s) + m) - zy;
      if (isn) ce = NAN;
      if (l32 == 0 && rvalid) {
        ce_sum += (double)ce;
        corr += (!isn && bi == y) ? 1u : 0u;
      }
    }
  }
  // reductions in a fixed order
  ce_sum += __shfl_xor(ce_sum, 32);
  corr += __shfl_xor(corr, 32);
  if (lane == 0) { red_ce[wave] = ce_sum; red_corr[wave] = corr; }
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    unsigned int cc = 0;
    for (int w = 0; w < NW; ++w) { t += red_ce[w]; cc += red_corr[w]; }
    a.part_ce[(size_t)v * a.n_chunks_total + a.chunk0 + chunk] = t;
    a.part_correct[(size_t)v * a.n_chunks_total + a.chunk0 + chunk] = cc;
  }
  vt_add(a.vtime, v, vt0);
}

// ---------------------------------------------- output layer, training in two passes
// The training step of the output layer (section 6.2), spread over many
// workgroups per variant instead of k_out's one.
// Pass 1, one workgroup per (32-row tile, variant): logits^T (classes x
// rows: a lane holds one row's classes crow(r) of its half, the row's other
// half in lane ^ 32; the four waves take quarters of the contraction,
// summed in a fixed order), then, as in k_out, per row max, NaN flag,
// log-sum-exp, CE, argmax (lowest index on ties, a NaN logit is a miss) and
// the gradient rows G = (softmax - onehot(y)) * scale, written out with the
// tile's sums of G by class, of CE and of hits.
template <typename S>
__global__ __launch_bounds__(256) void k_out_fwd(OutArgs<S> a) {
  using O = Op<S>;
  using F = typename O::Frag;
  constexpr int KM = O::KM, KE = O::KE;
  extern __shared__ __align__(16) char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, lh = lane >> 5;
  const int v = blockIdx.y, tile = blockIdx.x, ntile = a.Bp / 32;
  const uint64_t vt0 = vt_now();
  const int Kp = a.Kp, WS = Kp + O::PAD;
  float* red = reinterpret_cast<float*>(smem);          // [3][16][64] partial logits of waves 1-3; then G [32 rows][33]
  S* wop = reinterpret_cast<S*>(smem + 3 * 16 * 64 * 4);   // [32][WS]  W_L as operand, [class][k]
  const float* Wm = a.Wm + (size_t)v * 32 * Kp;
  {
    // sixteen float4 loads in flight per thread (the master is k-blocked [Kp/32][32][32])
    const int q = Kp / 4;                                // float4 per row
    for (int j0 = threadIdx.x; j0 < 32 * q; j0 += 256 * 16) {
      float4 w4[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int j = j0 + u * 256;
        w4[u] = j < 32 * q ? *reinterpret_cast<const float4*>(Wm + (size_t)j * 4) : make_float4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int j = j0 + u * 256;
        if (j < 32 * q) {
          S* dst = wop + ((j / 8) % 32) * WS + (j / 256) * 32 + (j % 8) * 4;   // row (j/8)%32, chunk j/256
          if constexpr (sizeof(S) == 2) {                 // four bf16 in one 8-byte write (WS * 2 is a multiple of 16)
            const uint32_t lo = (uint32_t)O::from_f32(w4[u].x) | (uint32_t)O::from_f32(w4[u].y) << 16;
            const uint32_t hi = (uint32_t)O::from_f32(w4[u].z) | (uint32_t)O::from_f32(w4[u].w) << 16;
            *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
          } else {
            dst[0] = O::from_f32(w4[u].x); dst[1] = O::from_f32(w4[u].y);
            dst[2] = O::from_f32(w4[u].z); dst[3] = O::from_f32(w4[u].w);
          }
        }
      }
    }
  }
  __syncthreads();
  const int steps = Kp / KM, s0 = wave * steps / 4, s1 = (wave + 1) * steps / 4;
  const S* ar = a.Arows + v * a.ar_vs + (size_t)(tile * 32 + l32) * Kp + lh * KE;
  const S* wr = wop + l32 * WS + lh * KE;
  f32x16_t acc0 = zero16(), acc1 = zero16();
  int st = s0;
  if constexpr (sizeof(S) == 4) {
    // fp32: within each 16 inputs, step u pairs inputs u (lanes 0-31) and
    // 8 + u (lanes 32-63): a lane's row operands are two 16-byte loads
    const float* ar8 = a.Arows + v * a.ar_vs + (size_t)(tile * 32 + l32) * Kp + 8 * lh;
    const float* wr8 = wop + l32 * WS + 8 * lh;
    for (; st + 8 <= s1; st += 8) {
      const int k = st * KM;                             // a multiple of 8 (Kp is a multiple of 32)
      const float4 x0 = *reinterpret_cast<const float4*>(ar8 + k);
      const float4 x1 = *reinterpret_cast<const float4*>(ar8 + k + 4);
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int u = 0; u < 8; u += 2) {
        acc0 = O::mma(wr8[k + u], xs[u], acc0);
        acc1 = O::mma(wr8[k + u + 1], xs[u + 1], acc1);
      }
    }
  }
  for (; st + 8 <= s1; st += 8) {                      // eight row loads in flight
    F x[8], w[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) { x[u] = O::load(ar + (st + u) * KM); w[u] = O::load(wr + (st + u) * KM); }
#pragma unroll
    for (int u = 0; u < 8; u += 2) {
      acc0 = O::mma(w[u], x[u], acc0);
      acc1 = O::mma(w[u + 1], x[u + 1], acc1);
    }
  }
  for (; st + 4 <= s1; st += 4) {
    F x[4], w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) { x[u] = O::load(ar + (st + u) * KM); w[u] = O::load(wr + (st + u) * KM); }
    acc0 = O::mma(w[0], x[0], acc0);
    acc1 = O::mma(w[1], x[1], acc1);
    acc0 = O::mma(w[2], x[2], acc0);
    acc1 = O::mma(w[3], x[3], acc1);
  }
  for (; st < s1; ++st) acc0 = O::mma(O::load(wr + st * KM), O::load(ar + st * KM), acc0);
  if (wave > 0) {
#pragma unroll
    for (int r = 0; r < 16; ++r) red[((wave - 1) * 16 + r) * 64 + lane] = acc0[r] + acc1[r];
  }
  __syncthreads();
  if (wave > 0) return;
  // lane: row rl = tile*32 + l32, classes c(r) = crow(r, lane), ascending in r
  const int C = a.C;
  const int rl = tile * 32 + l32;
  const int y = a.labels[rl];
  const bool rvalid = y >= 0;
  float z[16];
  float m = -INFINITY, bv = -INFINITY;
  int bi = 64, nanl = 0;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int c = crow(r, lane);
    const float zp = (((acc0[r] + acc1[r]) + red[r * 64 + lane]) + red[(16 + r) * 64 + lane]) + red[(32 + r) * 64 + lane];
    z[r] = zp + a.bias[(size_t)v * 32 + c];
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
  float ex[16], sl = 0.0f, zy = 0.0f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int c = crow(r, lane);
    ex[r] = c < C ? expf(z[r] - m) : 0.0f;
    sl += ex[r];
    if (c == y) zy = z[r];
  }
  const float sm = sl + __shfl_xor(sl, 32);
  zy += __shfl_xor(zy, 32);                          // exactly one lane of the pair holds class y
  float ce = (logf(sm) + m) - zy;
  if (nanl) ce = NAN;
  // G of this lane's classes: 4 consecutive classes per register group q
  float* gt = red;                                   // [32 rows][33] fp32 G for the class sums
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float g4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = 4 * q + j, c = crow(r, lane);
      const float sc = a.gscale ? a.gscale[((size_t)v * a.Bp + rl) * 32 + c] : a.scale;
      g4[j] = (c < C && rvalid) ? (ex[r] / sm - (c == y ? 1.0f : 0.0f)) * sc : 0.0f;
      gt[l32 * 33 + c] = g4[j];
    }
    S* gd = a.ogrd + ((size_t)v * a.Bp + rl) * 32 + 8 * q + 4 * lh;
    if constexpr (sizeof(S) == 2) {
      const uint32_t lo = (uint32_t)O::from_f32(g4[0]) | (uint32_t)O::from_f32(g4[1]) << 16;
      const uint32_t hi = (uint32_t)O::from_f32(g4[2]) | (uint32_t)O::from_f32(g4[3]) << 16;
      *reinterpret_cast<uint2*>(gd) = make_uint2(lo, hi);
    } else {
      *reinterpret_cast<float4*>(gd) = make_float4(g4[0], g4[1], g4[2], g4[3]);
    }
  }
  // the tile's sums: CE and hits over rows (lanes 0-31), G by class (lane c
  // sums column c in row order)
  double ce_sum = (lh == 0 && rvalid) ? (double)ce : 0.0;
  unsigned int corr = (lh == 0 && rvalid && !nanl && bi == y) ? 1u : 0u;
#pragma unroll
  for (int off = 16; off >= 1; off >>= 1) {
    ce_sum += __shfl_xor(ce_sum, off);
    corr += __shfl_xor(corr, off);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  const size_t ti = (size_t)v * ntile + tile;
  if (lh == 0) {
    float db = 0.0f;
    for (int rr = 0; rr < 32; ++rr) db += gt[rr * 33 + l32];
    a.opdb[ti * 32 + l32] = db;
  }
  if (lane == 0) { a.opce[ti] = ce_sum; a.opcorr[ti] = corr; }
  vt_add(a.vtime, v, vt0);
}

// Pass 2, one workgroup per (32-input column tile kt, variant): wave 0 forms
// dW_L[c][k] = sum_b G[b][c] A[k][b] for the tile's 32 inputs and applies
// the masked SGD update to those columns of the master; waves 1-3 form
// G_{L-1}[k][b] = (sum_c W_L[c][k] G[b][c]) * [A[k][b] > 0] for the same
// inputs from the columns' pre-update values, one 32-row batch tile at a
// time.  The kt == 0 workgroup also
// updates the biases and adds the CE and hit sums, tiles in order.  Each
// workgroup alone reads and writes its columns, so no other workgroup sees
// a half-updated W_L.
template <typename S, int BPMAX>
__global__ __launch_bounds__(256) void k_out_upd(OutArgs<S> a) {
  using O = Op<S>;
  constexpr int KM = O::KM, KE = O::KE;
  constexpr int GSTR = 32 + O::PAD, WSTR = 32 + O::PAD;
  constexpr int NG = BPMAX / KM;
  extern __shared__ __align__(16) char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, lh = lane >> 5;
  const int v = blockIdx.y, kt = blockIdx.x, ntile = a.Bp / 32;
  const uint64_t vt0 = vt_now();
  const int Kp = a.Kp;
  const int BT = a.Bp + O::PAD;
  float* stg = reinterpret_cast<float*>(smem);                       // [32][36] dW staging (wave 0)
  S* wold = reinterpret_cast<S*>(smem + 32 * 36 * 4);                // [32 classes][WSTR] old W_L columns
  S* gs = wold + 32 * WSTR;                                          // [Bp][GSTR] G rows
  S* gT = gs + (size_t)a.Bp * GSTR;                                  // [32 classes][BT] G columns
  // wave 0's operands for dW and the update, in flight with the G loads
  const S* Acv = a.Acols + v * a.ac_vs;
  const int nsteps = a.Bp / KM;
  const int rn = lane >> 1, cs = (lane & 1) * 16;
  typename O::Frag af[NG];
  float4 w4[4];
  uint32_t mw = 0;
  float* Wmv = a.Wm + (size_t)v * 32 * Kp;
  if (wave == 0) {
    if constexpr (sizeof(S) == 4) {
      // fp32: step s2 pairs batch rows s2 (lanes 0-31) and Bp/2 + s2 (lanes
      // 32-63), so a lane's operands are contiguous: four per 16-byte load
      const float* ap = Acv + (size_t)(kt * 32 + l32) * a.Bp + lh * (a.Bp / 2);
#pragma unroll
      for (int s4 = 0; s4 < NG; s4 += 4)
        if (s4 < nsteps) {
          const float4 x = *reinterpret_cast<const float4*>(ap + s4);
          af[s4] = x.x; af[s4 + 1] = x.y; af[s4 + 2] = x.z; af[s4 + 3] = x.w;
        }
    } else {
      const S* ap = Acv + (size_t)(kt * 32 + l32) * a.Bp + lh * KE;
#pragma unroll
      for (int s2 = 0; s2 < NG; ++s2)
        if (s2 < nsteps) af[s2] = O::load(ap + s2 * KM);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) w4[u] = *reinterpret_cast<const float4*>(Wmv + ((size_t)kt * 32 + rn) * 32 + cs + 4 * u);
    mw = a.mask[(size_t)v * 32 * (Kp / 32) + (size_t)rn * (Kp / 32) + kt];
  }
  {
    // 16-byte loads, all of a thread's issued before any is stored
    constexpr int PER = 16 / (int)sizeof(S);               // elements per 16 bytes
    const uint4* gsrc = reinterpret_cast<const uint4*>(a.ogrd + (size_t)v * a.Bp * 32);
    const int nvec = a.Bp * 32 / PER;                    // at most 256 * 32 / 4
    uint4 gv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = threadIdx.x + u * 256;
      gv[u] = i < nvec ? gsrc[i] : make_uint4(0, 0, 0, 0);
    }
    const float4 wv = reinterpret_cast<const float4*>(a.Wm + ((size_t)v * (Kp / 32) + kt) * 32 * 32)[threadIdx.x];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = threadIdx.x + u * 256;
      if (i < nvec) {
        const S* e = reinterpret_cast<const S*>(&gv[u]);
        const int row = (i * PER) >> 5, col = (i * PER) & 31;
        if constexpr (sizeof(S) == 2) {
          *reinterpret_cast<uint4*>(gs + row * GSTR + col) = gv[u];   // GSTR * 2 = 80 bytes: 16-byte aligned
        } else {
#pragma unroll
          for (int j = 0; j < PER; ++j) gs[row * GSTR + col + j] = e[j];
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) gT[(col + j) * BT + row] = e[j];
      }
    }
    // k-blocked master tile [c][32 k]: thread t holds class t / 8, inputs 4 (t % 8) .. +3
    S* wd = wold + (threadIdx.x >> 3) * WSTR + (threadIdx.x & 7) * 4;
    if constexpr (sizeof(S) == 2) {                     // WSTR * 2 = 80 bytes: 8-byte aligned pieces
      const uint32_t lo = (uint32_t)O::from_f32(wv.x) | (uint32_t)O::from_f32(wv.y) << 16;
      const uint32_t hi = (uint32_t)O::from_f32(wv.z) | (uint32_t)O::from_f32(wv.w) << 16;
      *reinterpret_cast<uint2*>(wd) = make_uint2(lo, hi);
    } else {
      wd[0] = O::from_f32(wv.x); wd[1] = O::from_f32(wv.y); wd[2] = O::from_f32(wv.z); wd[3] = O::from_f32(wv.w);
    }
  }
  __syncthreads();
  if (kt == 0) {
    const float lrv = a.lr[v];
    if (threadIdx.x < 32) {
      float db = 0.0f;
      for (int t = 0; t < ntile; ++t) db += a.opdb[((size_t)v * ntile + t) * 32 + threadIdx.x];
      const float bo = a.bias[(size_t)v * 32 + threadIdx.x];
      const bool bk = (a.bmask[v] >> threadIdx.x) & 1u;
      a.bias[(size_t)v * 32 + threadIdx.x] = bk ? __fsub_rn(bo, __fmul_rn(lrv, db)) : 0.0f;
    } else if (threadIdx.x == 64) {
      double t = 0.0;
      unsigned int cc = 0;
      for (int u = 0; u < ntile; ++u) { t += a.opce[(size_t)v * ntile + u]; cc += a.opcorr[(size_t)v * ntile + u]; }
      a.ce_acc[v] += t;
      a.correct_acc[v] += cc;
    }
  }
  if (wave == 0) {
    // dW tile staged in LDS, then lane (row rn, 16 columns) updates with float4
    const float lrv = a.lr[v];
    f32x16_t d = zero16();
#pragma unroll
    for (int s2 = 0; s2 < NG; ++s2)
      if (s2 < nsteps) {
        const int b = sizeof(S) == 4 ? lh * (a.Bp / 2) + s2 : s2 * KM + lh * KE;   // the pairing of af
        d = O::mma(O::load(&gT[l32 * BT + b]), af[s2], d);
      }
#pragma unroll
    for (int r = 0; r < 16; ++r) stg[crow(r, lane) * 36 + l32] = d[r];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    float wn[16];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float4 t = *reinterpret_cast<const float4*>(stg + rn * 36 + cs + 4 * u);
      const float dv[4] = {t.x, t.y, t.z, t.w};
      const float wv[4] = {w4[u].x, w4[u].y, w4[u].z, w4[u].w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool keep = (mw >> (cs + 4 * u + j)) & 1u;
        wn[4 * u + j] = keep ? __fsub_rn(wv[j], __fmul_rn(lrv, dv[j])) : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      *reinterpret_cast<float4*>(Wmv + ((size_t)kt * 32 + rn) * 32 + cs + 4 * u) =
          make_float4(wn[4 * u], wn[4 * u + 1], wn[4 * u + 2], wn[4 * u + 3]);
  }
  if (a.Gcols) {
    // gradient of the last hidden layer for inputs kt*32 .. +31, batch-contiguous, with ReLU'
    for (int bt = wave - 1; wave > 0 && bt < ntile; bt += 3) {   // waves 1-3 (wave 0 has dW)
      float av[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) av[r] = O::to_f32(Acv[(size_t)(kt * 32 + crow(r, lane)) * a.Bp + bt * 32 + l32]);
      f32x16_t acc = zero16();
#pragma unroll
      for (int ks = 0; ks < 32 / KM; ++ks) {
        const typename O::Frag wf = O::gather(&wold[(ks * KM + lh * KE) * WSTR + l32], WSTR);
        const typename O::Frag bf = O::load(&gs[(bt * 32 + l32) * GSTR + ks * KM + lh * KE]);
        acc = O::mma(wf, bf, acc);
      }
      const int b = bt * 32 + l32;
      S g[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        g[r] = O::from_f32(av[r] > 0.0f ? acc[r] : 0.0f);
        a.Gcols[v * a.gc_vs + (size_t)(kt * 32 + crow(r, lane)) * a.Bp + b] = g[r];
      }
      if (a.Grows) {
        // rows [b][k]: accumulator rows 4q..4q+3 are the consecutive inputs
        // kt 32 + 8q + 4 (l / 32) + 0..3, one 4-element store each
        S* gr = a.Grows + v * a.gr_vs + (size_t)b * Kp + kt * 32 + 4 * lh;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if constexpr (sizeof(S) == 2) {
            const uint32_t lo = (uint32_t)g[4 * q] | (uint32_t)g[4 * q + 1] << 16;
            const uint32_t hi = (uint32_t)g[4 * q + 2] | (uint32_t)g[4 * q + 3] << 16;
            *reinterpret_cast<uint2*>(gr + 8 * q) = make_uint2(lo, hi);
          } else {
            *reinterpret_cast<float4*>(gr + 8 * q) = make_float4(g[4 * q], g[4 * q + 1], g[4 * q + 2], g[4 * q + 3]);
          }
        }
      }
    }
  }
  vt_add(a.vtime, v, vt0);
}

// ------------------------------------------------------- hidden backward GEMM
// G_{l-1}[k][b] = (sum_n W_l[n][k] G_l[b][n]) * [A_{l-1}[k][b] > 0]; one
// 32x32 output tile per wave, operands straight from L2.
template <typename S>
__global__ __launch_bounds__(256) void k_bwd(BwdArgs<S> a) {
  using O = Op<S>;
  constexpr int KM = O::KM, KE = O::KE;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, lh = lane >> 5;
  const int v = blockIdx.y;
  const uint64_t vt0 = vt_now();
  const int tb = a.Bp / 32;
  const int t = blockIdx.x * 4 + wave;
  if (t >= (a.Kp / 32) * tb) return;
  const int kt = t / tb, bt = t % tb;
  const S* wr = a.Wt + (size_t)v * a.Kp * a.Np + (size_t)(kt * 32 + l32) * a.Np + lh * KE;
  const S* gr = a.Grows + v * a.gr_vs + (size_t)(bt * 32 + l32) * a.Np + lh * KE;
  f32x16_t acc = zero16();
  for (int n = 0; n < a.Np; n += KM) acc = O::mma(O::load(wr + n), O::load(gr + n), acc);
  const S* acv = a.Acols + v * a.ac_vs;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int k = kt * 32 + crow(r, lane);
    const int b = bt * 32 + l32;
    const float av = O::to_f32(acv[(size_t)k * a.Bp + b]);
    const S g = O::from_f32(av > 0.0f ? acc[r] : 0.0f);
    a.Gcols[v * a.gc_vs + (size_t)k * a.Bp + b] = g;
    if (a.Grows_out) a.Grows_out[v * a.go_vs + (size_t)b * a.Kp + k] = g;
  }
  vt_add(a.vtime, v, vt0);
}

// ------------------------------------------------------------- data movement
// rows[t][b][k] = X[perm[t*B + b]][k] (zero for k >= d0, b >= b_t, b >= B),
// labels[t][b] = y[...] or -1.
template <typename S>
__global__ __launch_bounds__(256) void k_gather(GatherArgs a) {
  using O = Op<S>;
  const int t = blockIdx.y, b = blockIdx.x;
  const int64_t r = (int64_t)t * a.B + b;
  const bool valid = b < a.B && r < a.n;
  const int64_t src = valid ? (a.perm ? (int64_t)a.perm[r] : r) : 0;
  S* rows = reinterpret_cast<S*>(a.rows) + (size_t)t * a.Bp * a.Kp;
  const float* x = a.X + src * a.d0;
  for (int k = threadIdx.x; k < a.Kp; k += blockDim.x) {
    const float xv = (valid && k < a.d0) ? x[k] : 0.0f;
    const int kp = a.res_order ? perm32(k & 31) : (k & 31);
    const size_t at = a.blocked ? ((size_t)(k >> 5) * a.Bp + b) * 32 + kp : (size_t)b * a.Kp + k;
    rows[at] = O::from_f32(xv);
  }
  if (threadIdx.x == 0) a.labels[(size_t)t * a.Bp + b] = valid ? a.y[src] : -1;
}

template <typename S>
__global__ __launch_bounds__(256) void k_transpose(TransposeArgs a) {
  __shared__ S tile[32][33];
  const int k0 = blockIdx.x * 32, b0 = blockIdx.y * 32, t = blockIdx.z;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const S* src = reinterpret_cast<const S*>(a.src) + (size_t)t * a.Bp * a.Kp;
  S* dst = reinterpret_cast<S*>(a.dst) + (size_t)t * a.Kp * a.Bp;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int b = b0 + ty + 8 * i;
    tile[ty + 8 * i][tx] = src[a.blocked ? ((size_t)blockIdx.x * a.Bp + b) * 32 + tx : (size_t)b * a.Kp + k0 + tx];
  }
  __syncthreads();
  // resident order: source position p holds input perm32(p); destination
  // column position c of each 32 rows holds batch row perm32(c)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int kk = ty + 8 * i;
    dst[(size_t)(k0 + kk) * a.Bp + b0 + tx] = a.res_order ? tile[perm32(tx)][perm32(kk)] : tile[tx][kk];
  }
}

// W1 master of a two-layer net between the k-blocked layout [P][Kp/32][Hp][32]
// and the register image the fused training kernel streams: in block kb, wave
// w (hidden units 32w..32w+31) reads 4 KiB as [q][lane][4], where lane
// l32 + 32 lh holds inputs 8q + 4lh + 0..3 of unit 32w + l32.  One thread
// moves one 16-byte group; to_image = 1 converts blocked -> image.
__global__ __launch_bounds__(256) void k_w1_image(const float* __restrict__ src, float* __restrict__ dst,
                                                  int64_t groups, int Hp, int to_image) {
  for (int64_t gi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; gi < groups;
       gi += (int64_t)gridDim.x * blockDim.x) {
    // gi enumerates the image: ((((v * nkb + kb) * NW + w) * 4 + q) * 64 + lane)
    const int lane = (int)(gi & 63), q = (int)((gi >> 6) & 3);
    const int64_t blk = gi >> 8;                     // (v * nkb + kb) * NW + w
    const int NW = Hp / 32, w = (int)(blk % NW);
    const int64_t vkb = blk / NW;                    // v * nkb + kb
    const int n = 32 * w + (lane & 31), kl = 8 * q + 4 * (lane >> 5);
    const int64_t img = gi * 4, kblk = (vkb * Hp + n) * 32 + kl;
    const float4 val = *reinterpret_cast<const float4*>(src + (to_image ? kblk : img));
    *reinterpret_cast<float4*>(dst + (to_image ? img : kblk)) = val;
  }
}

// W1 mask words of a two-layer net from row words [P][Hp][Kp/32] to
// block-major words [P][Kp/32][Hp] (the fused kernel's per-block read is contiguous).
__global__ __launch_bounds__(256) void k_mask_block_major(const uint32_t* __restrict__ src,
                                                          uint32_t* __restrict__ dst, int64_t words, int Hp,
                                                          int nkb) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int n = (int)(i % Hp);
    const int64_t vkb = i / Hp;                      // v * nkb + kb
    const int64_t v = vkb / nkb, kb = vkb % nkb;
    dst[i] = src[(v * Hp + n) * nkb + kb];
  }
}

__global__ __launch_bounds__(256) void k_zero(uint32_t* p, size_t words) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

__global__ __launch_bounds__(256) void k_reduce_partials(const double* part_ce, const unsigned int* part_corr,
                                                         int P, int nch, double* ce_out,
                                                         unsigned long long* corr_out) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= P) return;
  double s = 0.0;
  unsigned long long c = 0;
  for (int i = 0; i < nch; ++i) {
    s += part_ce[(size_t)v * nch + i];
    c += part_corr[(size_t)v * nch + i];
  }
  ce_out[v] = s;
  corr_out[v] = c;
}

// ---------------------------------------------------------------- launchers
static inline unsigned grid_for(int64_t items, int per_block = 256, int64_t cap = 65536) {
  int64_t g = (items + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

hipError_t launch_init(const InitArgs& a, hipStream_t s, const LaunchEv& ev) {
  const int64_t items = (int64_t)a.P * a.Np * (a.Kp / 32);
  hipExtLaunchKernelGGL(k_init, dim3(grid_for(items)), dim3(256), 0, s, ev.start, ev.stop, 0, a);
  return hipGetLastError();
}

size_t layer_stage_bytes() { return (size_t)4 * 32 * 36 * 4; }

int layer_block_cols(int Kp, int elt, int pad) {
  const size_t stage = layer_stage_bytes();
  int cap = (int)((kLayerLds - stage) / (32 * (size_t)elt)) - pad;
  cap = cap / 32 * 32;
  const int nblk = (Kp + cap - 1) / cap;
  return round_up((Kp + nblk - 1) / nblk, 32);
}

template <typename S>
hipError_t launch_layer(const LayerArgs<S>& a0, int P, hipStream_t s, const LaunchEv& ev) {
  LayerArgs<S> a = a0;
  a.KB = layer_block_cols(a.Kp, (int)sizeof(S), Op<S>::PAD);
  const size_t lds = (size_t)32 * (a.KB + Op<S>::PAD) * sizeof(S) + layer_stage_bytes();
  const dim3 grid(a.Np / 32, P);
  if (a.Bp <= 128 || !a.do_update) {
    static bool attr = false;
    if (!attr) {
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_layer<S, 128>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLayerLds);
      attr = true;
    }
    hipExtLaunchKernelGGL((k_layer<S, 128>), grid, dim3(256), lds, s, ev.start, ev.stop, 0, a);
  } else {
    static bool attr = false;
    if (!attr) {
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_layer<S, 256>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLayerLds);
      attr = true;
    }
    hipExtLaunchKernelGGL((k_layer<S, 256>), grid, dim3(256), lds, s, ev.start, ev.stop, 0, a);
  }
  return hipGetLastError();
}

template <typename S>
hipError_t launch_out(const OutArgs<S>& a, int P, hipStream_t s, const LaunchEv& ev) {
  if (a.train) {
    // two passes: rows of the batch, then columns of W_L
    if (!a.ogrd || !a.opdb || !a.opce || !a.opcorr || a.Bp > 256 || a.Bp % 32 || a.Kp % 32) return hipErrorInvalidValue;
    const size_t lds1 = (size_t)3 * 16 * 64 * 4 + (size_t)32 * (a.Kp + Op<S>::PAD) * sizeof(S);
    const size_t lds2 = (size_t)32 * 36 * 4 + (size_t)32 * (32 + Op<S>::PAD) * sizeof(S) +
                        (size_t)a.Bp * (32 + Op<S>::PAD) * sizeof(S) + (size_t)32 * (a.Bp + Op<S>::PAD) * sizeof(S);
    if (lds1 > kLdsBudget || lds2 > kLdsBudget) return hipErrorInvalidValue;
    static bool attr = false;
    if (!attr) {
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_out_fwd<S>), hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)kLdsBudget);
      attr = true;
    }
    hipExtLaunchKernelGGL(k_out_fwd<S>, dim3(a.Bp / 32, P), dim3(256), lds1, s, ev.start, nullptr, 0, a);
    if (a.Bp <= 128)
      hipExtLaunchKernelGGL((k_out_upd<S, 128>), dim3(a.Kp / 32, P), dim3(256), lds2, s, nullptr, ev.stop, 0, a);
    else
      hipExtLaunchKernelGGL((k_out_upd<S, 256>), dim3(a.Kp / 32, P), dim3(256), lds2, s, nullptr, ev.stop, 0, a);
    return hipGetLastError();
  }
  const size_t lds = (size_t)32 * (a.Kp + Op<S>::PAD) * sizeof(S);
  if (lds > kLdsBudget) return hipErrorInvalidValue;
  const dim3 grid((a.rows + kOutRows - 1) / kOutRows, P);
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_out<S>), hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)kLdsBudget);
    attr = true;
  }
  hipExtLaunchKernelGGL(k_out<S>, grid, dim3(64 * kOutWaves), lds, s, ev.start, ev.stop, 0, a);
  return hipGetLastError();
}

template <typename S>
hipError_t launch_bwd(const BwdArgs<S>& a, int P, hipStream_t s, const LaunchEv& ev) {
  const int tiles = (a.Kp / 32) * (a.Bp / 32);
  hipExtLaunchKernelGGL(k_bwd<S>, dim3((tiles + 3) / 4, P), dim3(256), 0, s, ev.start, ev.stop, 0, a);
  return hipGetLastError();
}

template <typename S>
hipError_t launch_gather(const GatherArgs& a, hipStream_t s, const LaunchEv& ev) {
  hipExtLaunchKernelGGL(k_gather<S>, dim3(a.Bp, a.T), dim3(256), 0, s, ev.start, ev.stop, 0, a);
  return hipGetLastError();
}

template <typename S>
hipError_t launch_transpose(const TransposeArgs& a, hipStream_t s, const LaunchEv& ev) {
  hipExtLaunchKernelGGL(k_transpose<S>, dim3(a.Kp / 32, a.Bp / 32, a.T), dim3(256), 0, s, ev.start, ev.stop, 0, a);
  return hipGetLastError();
}

hipError_t launch_zero_bytes(void* p, size_t bytes, hipStream_t s, const LaunchEv& ev) {
  const size_t words = bytes / 4;
  if (words == 0) return hipSuccess;
  hipExtLaunchKernelGGL(k_zero, dim3(grid_for((int64_t)words, 256, 4096)), dim3(256), 0, s, ev.start, ev.stop, 0,
                        (uint32_t*)p, words);
  return hipGetLastError();
}

hipError_t launch_w1_image(const float* src, float* dst, int P, int Kp, int Hp, bool to_image, hipStream_t s,
                           const LaunchEv& ev) {
  const int64_t groups = (int64_t)P * Kp * Hp / 4;
  hipExtLaunchKernelGGL(k_w1_image, dim3(grid_for(groups, 256, 16384)), dim3(256), 0, s, ev.start, ev.stop, 0, src,
                        dst, groups, Hp, to_image ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_mask_block_major(const uint32_t* src, uint32_t* dst, int P, int Kp, int Hp, hipStream_t s,
                                   const LaunchEv& ev) {
  const int64_t words = (int64_t)P * Hp * (Kp / 32);
  hipExtLaunchKernelGGL(k_mask_block_major, dim3(grid_for(words, 256, 16384)), dim3(256), 0, s, ev.start, ev.stop,
                        0, src, dst, words, Hp, Kp / 32);
  return hipGetLastError();
}

// Exhaustive check of the packed bf16 conversion the kernels use against the
// bit-level rounding, over every binary32 encoding in two pairings of the
// instruction's operands: counts[0] for (i, i | 2^31), counts[1] for
// (2j, 2j + 1), i, j < 2^31, each the number of differing halves.
__global__ __launch_bounds__(256) void k_bf16_check(unsigned long long* counts) {
  const uint64_t nthreads = (uint64_t)gridDim.x * 256;
  unsigned long long c[2] = {0, 0};
  for (uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x; i < (1ull << 32); i += nthreads) {
    const uint32_t j = (uint32_t)(i & 0x7fffffffu), pairing = (uint32_t)(i >> 31);
    const uint32_t e0 = pairing ? 2u * j : j, e1 = pairing ? 2u * j + 1u : j | 0x80000000u;
    const float f[2] = {__uint_as_float(e0), __uint_as_float(e1)};
    uint32_t p[1];
    to_bf16x2(f, p);
    c[pairing] += ((uint16_t)p[0] != f32_to_bf16_bits(f[0])) + ((uint16_t)(p[0] >> 16) != f32_to_bf16_bits(f[1]));
  }
  if (c[0]) atomicAdd(&counts[0], c[0]);
  if (c[1]) atomicAdd(&counts[1], c[1]);
}

hipError_t launch_bf16_check(unsigned long long* counts, hipStream_t s) {
  hipLaunchKernelGGL(k_bf16_check, dim3(4096), dim3(256), 0, s, counts);
  return hipGetLastError();
}

hipError_t launch_reduce_partials(const double* part_ce, const unsigned int* part_corr, int P, int n_chunks,
                                  double* ce_out, unsigned long long* corr_out, hipStream_t s, const LaunchEv& ev) {
  hipExtLaunchKernelGGL(k_reduce_partials, dim3((P + 255) / 256), dim3(256), 0, s, ev.start, ev.stop, 0, part_ce,
                        part_corr, P, n_chunks, ce_out, corr_out);
  return hipGetLastError();
}

template hipError_t launch_layer<float>(const LayerArgs<float>&, int, hipStream_t, const LaunchEv&);
template hipError_t launch_layer<uint16_t>(const LayerArgs<uint16_t>&, int, hipStream_t, const LaunchEv&);
template hipError_t launch_out<float>(const OutArgs<float>&, int, hipStream_t, const LaunchEv&);
template hipError_t launch_out<uint16_t>(const OutArgs<uint16_t>&, int, hipStream_t, const LaunchEv&);
template hipError_t launch_bwd<float>(const BwdArgs<float>&, int, hipStream_t, const LaunchEv&);
template hipError_t launch_bwd<uint16_t>(const BwdArgs<uint16_t>&, int, hipStream_t, const LaunchEv&);
template hipError_t launch_gather<float>(const GatherArgs&, hipStream_t, const LaunchEv&);
template hipError_t launch_gather<uint16_t>(const GatherArgs&, hipStream_t, const LaunchEv&);
template hipError_t launch_transpose<float>(const TransposeArgs&, hipStream_t, const LaunchEv&);
template hipError_t launch_transpose<uint16_t>(const TransposeArgs&, hipStream_t, const LaunchEv&);

}  // namespace gevo
