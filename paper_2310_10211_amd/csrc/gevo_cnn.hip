// Convolutional prediction workload (section 4.3: the prediction workload
// runs a model over a dataset and records its error; Table 1 lists MobileNet,
// a depthwise-separable convolutional net, among the models): P variants of a
// CIFAR-shaped MobileNet-like net, each the caller's base weights times
// fl(1 + fl(std eps)) under its own Bernoulli(rho_v) mask (section 4.2's
// pruning edits, as in the fully connected workload 4), evaluated over a test
// set.  Per 64-image chunk and for all variants at once:
//   stem   3x3 convolution, stride 1, zero padding 1, bias, ReLU  (k_cnn_stem)
//   block  3x3 depthwise convolution, stride 1|2, bias, ReLU      (k_cnn_dw)
//          1x1 pointwise convolution = a per-variant GEMM over the
//          chunk's pixels, bias, ReLU                             (k_fwd_gemm)
//          (a pointwise layer and the next block's depthwise layer
//          run as one kernel when its map fits LDS strips)        (k_cnn_pwdw)
//   head   global average pooling                                 (k_cnn_pool)
//          fully connected layer, softmax cross-entropy, argmax   (k_out)
// bf16 operands and activations, fp32 accumulation, fp32 master weights.
#include "gevo_internal.h"
#include "gevo_device.h"
#include "gevo.h"

#include <hip/hip_ext.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

namespace gevo {

namespace {

constexpr int kCnnChunk = 64;            // images per prediction chunk

struct CnnStemArgs {
  const float* x; int64_t n_test; int img0;   // test images [n][H][W][C] fp32, first image of the chunk
  int H, W;
  int Np;                                     // output channels
  uint32_t w_magic, w2_magic;                 // ceil(2^32 / W), ceil(2^32 / (W + 2)): exact quotients below 2^16
  const float* wp; const float* bias;         // bf16-valued taps [P][9C][Np] (fp32 storage), biases [P][Np]
  uint16_t* out; size_t out_vs;               // [v][chunk][H][W][Np] bf16
};

struct CnnDwArgs {
  const uint16_t* in; size_t in_vs;           // [v][chunk][H][W][C]
  uint16_t* out; size_t out_vs;               // [v][chunk][Ho][Wo][C]
  int H, W, C, Ho, Wo, stride;
  const uint32_t* wp; const float* bias;      // tap pairs [P][5][C] (bf16 x 2), biases [P][C]
};

struct CnnPwDwArgs {
  const uint16_t* in; size_t in_vs;           // pointwise input [v][chunk][H][W][Cin]
  const float* Wm; const float* pbias;        // pointwise master [P][Cin/32][Cout][32], biases [P][Cout]
  const uint32_t* dwp; const float* dbias;    // depthwise tap pairs [P][5][Cout] (bf16 x 2), biases [P][Cout]
  uint16_t* out; size_t out_vs;               // depthwise output [v][chunk][Ho][Wo][Cout]
  int H, W, Cin, Cout, Ho, Wo, R;             // R: depthwise output rows per strip
  int ipw;                                    // images per workgroup (divides the chunk)
  uint32_t wo_magic, c8in_magic;              // ceil(2^32 / Wo), ceil(2^32 / (Cin / 8)): exact quotients below 2^16
};

struct CnnPoolArgs {
  const uint16_t* in; size_t in_vs;           // [v][chunk][HW][C]
  int HW, C;
  uint16_t* out; size_t out_vs;               // [v][chunk][C]
};

__device__ __forceinline__ float bf16r(float f) { return bf16_bits_to_f32(f32_to_bf16_bits(f)); }

}  // namespace

// Prediction copy of one weight tensor: out[v][k][n] = bf16(W_v[k][n]) held in
// fp32, read from the k-blocked master [v][Kp/32][Np][32].  The handle never
// changes its masters, so this runs once, at init.
__global__ __launch_bounds__(256) void k_cnn_pack(const float* __restrict__ Wm, int Kp, int Np, int K, int N, int P,
                                                  float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)P * K * N) return;
  const int n = (int)(i % N), k = (int)((i / N) % K), v = (int)(i / ((int64_t)K * N));
  out[i] = bf16r(Wm[(size_t)v * Np * Kp + ((size_t)(k / 32) * Np + n) * 32 + k % 32]);
}

// Workgroup slot -> (variant, tile): slot i runs on XCD i % 8, and each XCD
// takes a contiguous range of the variants' tiles in order, so neighbouring
// tiles (which share input rows) meet in the same L2.
__device__ __forceinline__ void cnn_slot(int& v, int& tile) {
  const int gx = gridDim.x, total = gx * gridDim.y, i = blockIdx.y * gx + blockIdx.x;
  const int j = total % 8 == 0 ? (i % 8) * (total / 8) + i / 8 : i;
  v = j / gx;
  tile = j % gx;
}

typedef uint32_t cnn_u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16_t cnn_mma(cnn_u32x4 a, cnn_u32x4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}

// Depthwise taps of the prediction copy as bf16 pairs: out[v][p][c] holds taps
// 2p (low half) and 2p + 1 (high half) of channel c, the high half of pair 4
// being zero, read from the k-blocked master [v][1][C][32] (taps k < 9 of
// channel c).
__global__ __launch_bounds__(256) void k_cnn_pack_pairs(const float* __restrict__ Wm, int C, int P,
                                                        uint32_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)P * 5 * C) return;
  const int c = (int)(i % C), p = (int)((i / C) % 5), v = (int)(i / ((int64_t)5 * C));
  const float* w = Wm + ((size_t)v * C + c) * 32;
  const uint32_t lo = f32_to_bf16_bits(w[2 * p]);
  const uint32_t hi = 2 * p + 1 < 9 ? f32_to_bf16_bits(w[2 * p + 1]) : 0u;
  out[i] = lo | hi << 16;
}

// A removed block layer in its identity form, written over one variant's
// master (k-blocked [Kp/32][Np][32]), biases [Np] and mask bits ([Np][Kp/32],
// bit k % 32 of word k / 32): W[k][n] = 1 where k == centre (a depthwise
// layer's centre tap, for every channel) or, with centre < 0, where k == n (a
// pointwise layer: channels passed on, the first N kept); every other weight
// and the padding +0, every bias +0 except those of the channels a widening
// pointwise layer appends, which are 1 (the value section 4.1 pads tensors
// with: relu(0 + 1) = 1).  Every block layer reads a ReLU output, so
// relu(x 1 + 0) = x exactly and the layer passes its input on.
__global__ __launch_bounds__(256) void k_cnn_identity(float* __restrict__ Wm, float* __restrict__ bias,
                                                      uint32_t* __restrict__ mask, int Kp, int Np, int K, int N,
                                                      int centre) {
  const int stride = gridDim.x * blockDim.x, t0 = blockIdx.x * blockDim.x + threadIdx.x;
  auto one = [&](int k, int n) { return k < K && n < N && (centre >= 0 ? k == centre : k == n); };
  for (int i = t0; i < Kp * Np; i += stride) {
    const int kb = i / (Np * 32), r = i - kb * Np * 32, n = r / 32, k = kb * 32 + r % 32;
    Wm[i] = one(k, n) ? 1.0f : 0.0f;
  }
  for (int i = t0; i < Np * (Kp / 32); i += stride) {
    const int n = i / (Kp / 32), kw = i - n * (Kp / 32);
    uint32_t bits = 0;
    for (int b = 0; b < 32; ++b) bits |= one(32 * kw + b, n) ? 1u << b : 0u;
    mask[i] = bits;
  }
  for (int n = t0; n < Np; n += stride) bias[n] = (centre < 0 && n >= K && n < N) ? 1.0f : 0.0f;
}

typedef __bf16 cnn_bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float cnn_dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(cnn_bf16x2, a), __builtin_bit_cast(cnn_bf16x2, b), c,
                                         false);
}

// One depthwise output for 8 channels: acc[j] += sum_t in[t][j] w[t][j] over
// the 9 taps (in[t]: 8 bf16 channels of tap t = 3 dy + dx, zero outside the
// image).  Taps go in pairs (2p, 2p + 1) through the bf16 dot2 instruction
// (two products summed into the fp32 accumulator), the inputs re-paired by
// channel.  tap(t) gives in[t]; wp: tap pairs [5][C] at this thread's first
// channel.
template <typename Tap>
__device__ __forceinline__ void cnn_dw_dot(Tap tap, const uint32_t* wp, int C, float (&acc)[8]) {
#pragma unroll
  for (int p = 0; p < 5; ++p) {
    const uint4 wa = *reinterpret_cast<const uint4*>(wp + p * C);
    const uint4 wb = *reinterpret_cast<const uint4*>(wp + p * C + 4);
    const uint32_t w[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
    const uint4 q0 = tap(2 * p);
    const uint4 q1 = p < 4 ? tap(2 * p + 1) : make_uint4(0, 0, 0, 0);
    const uint32_t a0[4] = {q0.x, q0.y, q0.z, q0.w}, a1[4] = {q1.x, q1.y, q1.z, q1.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {                       // channels 2i, 2i + 1
      // byte permutes of {a1 (bytes 4-7), a0 (bytes 0-3)}: lo = channel 2i of
      // taps 2p, 2p + 1; hi = channel 2i + 1 of both
      const uint32_t lo = __builtin_amdgcn_perm(a1[i], a0[i], 0x05040100u);
      const uint32_t hi = __builtin_amdgcn_perm(a1[i], a0[i], 0x07060302u);
      acc[2 * i] = cnn_dot2(lo, w[2 * i], acc[2 * i]);
      acc[2 * i + 1] = cnn_dot2(hi, w[2 * i + 1], acc[2 * i + 1]);
    }
  }
}

// stem as a GEMM on the matrix cores: per 32-pixel tile and 32 output
// channels, out^T[n][p] = sum_k W[k][n] patch_p[k] with the taps k = (3 dy + dx)
// C + c padded with zeros to a multiple of 16 (32x32x16 bf16 MFMAs, fp32
// accumulation).  Lane l gives column (pixel) l % 32 and k slots 8 (l / 32)
// + 0..7 of each 16-k step in both operands; the accumulator holds channels
// crow(r, l) of pixel l % 32.  One workgroup per (variant, image): the image,
// rounded to bf16 and zero-padded by one pixel, sits in LDS; each wave stages
// its 32 x 32 results in LDS and stores them as whole 64-byte pixel rows.
template <int C>
__global__ __launch_bounds__(256) void k_cnn_stem(CnnStemArgs a) {
  constexpr int K = 9 * C, KS = (K + 15) / 16;
  __shared__ __align__(16) uint32_t stage[4][32 * 20];         // per wave: 32 pixels x 32 channels bf16 (+8 pad)
  extern __shared__ __align__(16) uint16_t im[];                // [H + 2][W + 2][C]
  int v, img;
  cnn_slot(v, img);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l32 = lane & 31, lh = lane >> 5;
  const int H = a.H, W = a.W, W2 = W + 2, HW = H * W, Np = a.Np;
  const int64_t g = (int64_t)a.img0 + img;
  const bool valid = g < a.n_test;
  for (int i = threadIdx.x; i < (H + 2) * W2 * C; i += blockDim.x) {
    const int c = i % C, pix = i / C, py = (int)__umulhi((uint32_t)pix, a.w2_magic);
    const int yy = py - 1, xx = pix - py * W2 - 1;
    const bool in = valid && yy >= 0 && yy < H && xx >= 0 && xx < W;
    const int64_t at = in ? ((g * H + yy) * W + xx) * C + c : 0;   // in-bounds even when unused
    im[i] = in ? f32_to_bf16_bits(a.x[at]) : (uint16_t)0;
  }
  const float* wv = a.wp + (size_t)v * K * Np;
  const float* bv = a.bias + (size_t)v * Np;
  uint16_t* ov = a.out + a.out_vs * v + (size_t)img * HW * Np;
  uint32_t* st = stage[wave];
  __syncthreads();
  // tap k of this lane half: LDS offset relative to the pixel's top-left neighbour
  int toff[KS][8];
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k0 = 16 * s + j, k1 = k0 + 8;
      const int t0 = k0 < K ? ((k0 / C) / 3 * W2 + (k0 / C) % 3) * C + k0 % C : -1;
      const int t1 = k1 < K ? ((k1 / C) / 3 * W2 + (k1 / C) % 3) * C + k1 % C : -1;
      toff[s][j] = lh ? t1 : t0;
    }
  const int ntiles = (HW + 31) / 32;
  for (int n0 = 0; n0 < Np; n0 += 32) {
    // A operand (taps of channels n0 + l32) and the biases of this lane's accumulator rows
    cnn_u32x4 aq[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      uint32_t hw[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = 16 * s + 8 * lh + j;
        hw[j] = k < K ? f32_to_bf16_bits(wv[(size_t)k * Np + n0 + l32]) : 0u;
      }
      aq[s] = cnn_u32x4{hw[0] | hw[1] << 16, hw[2] | hw[3] << 16, hw[4] | hw[5] << 16, hw[6] | hw[7] << 16};
    }
    float bias[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) bias[r] = bv[n0 + crow(r, lane)];
    for (int t = wave; t < ntiles; t += 4) {
      const int p = min(t * 32 + l32, HW - 1);           // pixels past the image: computed, never stored
      const int py = (int)__umulhi((uint32_t)p, a.w_magic);    // p / W
      const int base = (py * W2 + (p - py * W)) * C;
      f32x16_t acc = zero16();
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        uint32_t hv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) hv[j] = toff[s][j] >= 0 ? (uint32_t)im[base + toff[s][j]] : 0u;
        const cnn_u32x4 bq{hv[0] | hv[1] << 16, hv[2] | hv[3] << 16, hv[4] | hv[5] << 16, hv[6] | hv[7] << 16};
        acc = cnn_mma(aq[s], bq, acc);
      }
      float f[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float z = acc[r] + bias[r];
        f[r] = z > 0.0f ? z : 0.0f;
      }
      uint32_t pk[8];
      to_bf16x2(f, pk);                                  // pk[i]: channels crow(2i), crow(2i) + 1
#pragma unroll
      for (int i = 0; i < 8; ++i) st[l32 * 20 + crow(2 * i, lane) / 2] = pk[i];
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int h = 0; h < 2; ++h) {                      // 16 pixels x 64 bytes per pass
        const int px = 16 * h + (lane >> 2), q = lane & 3;
        const cnn_u32x4 val = *reinterpret_cast<const cnn_u32x4*>(st + px * 20 + q * 4);
        if (t * 32 + px < HW) *reinterpret_cast<cnn_u32x4*>(ov + (size_t)(t * 32 + px) * Np + n0 + q * 8) = val;
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
}

// depthwise 3x3 with stride S: one thread per (image, output column, 8
// channels) of one variant, walking down the output rows with the 3 x 3 input
// window in registers (a new output row loads S new input rows of three
// pixels).  A wave's loads and stores cover 8 whole 16-byte channel groups of
// consecutive pixels.
template <int S>
__global__ __launch_bounds__(256) void k_cnn_dw(CnnDwArgs a) {
  extern __shared__ uint32_t dl[];                     // tap pairs [5][C], then bias [C] (fp32)
  int v, w;
  cnn_slot(v, w);
  const int C = a.C, H = a.H, W = a.W;
  const uint32_t* wv = a.wp + (size_t)v * 5 * C;
  for (int i = threadIdx.x; i < 5 * C; i += blockDim.x) dl[i] = wv[i];
  float* dbias = reinterpret_cast<float*>(dl + 5 * C);
  for (int c = threadIdx.x; c < C; c += blockDim.x) dbias[c] = a.bias[(size_t)v * C + c];
  __syncthreads();
  const int C8 = C / 8;
  const int i = w * 256 + threadIdx.x;
  if (i >= kCnnChunk * a.Wo * C8) return;
  const int c0 = (i % C8) * 8, xo = (i / C8) % a.Wo, img = i / (C8 * a.Wo);
  const uint16_t* src = a.in + a.in_vs * v + (size_t)img * H * W * C + c0;
  uint16_t* dst = a.out + a.out_vs * v + (size_t)img * a.Ho * a.Wo * C + (size_t)xo * C + c0;
  const int x0 = S * xo - 1;
  uint4 win[3][3];                                     // [input row of the window][column]
  auto load_row = [&](int r, uint4 (&row)[3]) {
#pragma unroll
    for (int dx = 0; dx < 3; ++dx) {
      const int xx = x0 + dx;
      const bool in = r >= 0 && r < H && xx >= 0 && xx < W;
      row[dx] = in ? *reinterpret_cast<const uint4*>(src + ((size_t)r * W + xx) * C) : make_uint4(0, 0, 0, 0);
    }
  };
  load_row(-1, win[0]);
  load_row(0, win[1]);
  load_row(1, win[2]);
  const float* bias = dbias + c0;
  for (int yo = 0; yo < a.Ho; ++yo) {
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
    cnn_dw_dot([&](int t) { return win[t / 3][t % 3]; }, dl + c0, C, acc);
    float f[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float z = acc[j] + bias[j];
      f[j] = z > 0.0f ? z : 0.0f;
    }
    uint32_t pk[4];
    to_bf16x2(f, pk);
    *reinterpret_cast<uint4*>(dst + (size_t)yo * a.Wo * C) = make_uint4(pk[0], pk[1], pk[2], pk[3]);
    // window of output row yo + 1: input rows S (yo + 1) - 1 .. + 2
    const int r0 = S * (yo + 1) - 1;
    if (S == 1) {
#pragma unroll
      for (int dx = 0; dx < 3; ++dx) {
        win[0][dx] = win[1][dx];
        win[1][dx] = win[2][dx];
      }
      load_row(r0 + 2, win[2]);
    } else {
#pragma unroll
      for (int dx = 0; dx < 3; ++dx) win[0][dx] = win[2][dx];
      load_row(r0 + 1, win[1]);
      load_row(r0 + 2, win[2]);
    }
  }
}

// A pointwise convolution fused with the depthwise convolution after it
// (stride S): one workgroup per (variant, ipw images) walks each image's
// depthwise output rows in strips of R (several images per workgroup share
// one load of the variant's pointwise weights).  A strip needs the pointwise outputs of S (R - 1) + 3
// input rows (those inside the image):
//   1. their pointwise inputs are staged in LDS (rows of the image are
//      contiguous, so these are whole 16-byte pieces of one contiguous span;
//      the next strip's pieces are loaded into registers during the current
//      strip's pointwise phase and stored to LDS before its depthwise phase,
//      whose global stores would otherwise join the wait);
//   2. the pointwise outputs go to LDS as bf16 from 32x32x16 bf16 MFMAs with
//      fp32 accumulation: per 32-pixel x 32-channel tile out^T[n][p] =
//      sum_k W[k][n] A[p][k]; lane l gives channel / pixel l % 32 and k slots
//      8 (l / 32) + 0..7 of each 16-k step in both operands, and its
//      accumulator holds channels crow(r, l) of pixel l % 32; wave w takes
//      the channel tiles w, w + 4, ...;
//   3. the depthwise convolution reads them from LDS, one thread per (output
//      pixel, 8 channels), and writes its output.
// The pointwise output never goes to global memory.  Cin <= 128, Cout = 128 NT,
// and a
// strip's inputs are at most kPwDwPieces x 256 pieces of 16 bytes.
constexpr int kPwDwPieces = 8;

template <int S, int NT>
__global__ __launch_bounds__(256, NT == 1 ? 2 : 1) void k_cnn_pwdw(CnnPwDwArgs a) {
  extern __shared__ __align__(16) char smem[];
  int v, w;
  cnn_slot(v, w);
  const int Cin = a.Cin, Cout = a.Cout, H = a.H, W = a.W, KS = Cin / 16, AS = Cin + 8, PS = Cout + 8;
  const int rows_in = S * (a.R - 1) + 3;
  uint16_t* al = reinterpret_cast<uint16_t*>(smem);                                // [rows_in W][Cin + 8]
  uint16_t* pl = al + (((size_t)rows_in * W * AS + 7) & ~(size_t)7);                 // [rows_in][W][Cout + 8]
  uint32_t* dt = reinterpret_cast<uint32_t*>(pl + (((size_t)rows_in * W * PS + 7) & ~(size_t)7));  // [5][Cout] pairs
  float* dbias = reinterpret_cast<float*>(dt + 5 * Cout);                                             // [Cout]
  for (int i = threadIdx.x; i < 5 * Cout; i += blockDim.x) dt[i] = a.dwp[(size_t)v * 5 * Cout + i];
  for (int c = threadIdx.x; c < Cout; c += blockDim.x) dbias[c] = a.dbias[(size_t)v * Cout + c];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l32 = lane & 31, lh = lane >> 5;
  const float* Wv = a.Wm + (size_t)v * Cin * Cout;
  const float* pb = a.pbias + (size_t)v * Cout;
  const int C8in = Cin / 8;
  // jobs: (image, strip) pairs of this workgroup's images, in order
  const int nstrips = (a.Ho + a.R - 1) / a.R, njobs = a.ipw * nstrips;
  auto job_image = [&](int j) { return w * a.ipw + j / nstrips; };
  auto job_row = [&](int j) { return (j % nstrips) * a.R; };
  // rows [rv0, rv1) of the strip starting at depthwise output row yo0
  auto strip_rows = [&](int yo0, int& rv0, int& rv1) {
    rv0 = max(0, S * yo0 - 1);
    rv1 = min(H, S * yo0 - 1 + rows_in);
  };
  cnn_u32x4 pre[kPwDwPieces];
  auto fetch = [&](int j) {
    int rv0, rv1;
    strip_rows(job_row(j), rv0, rv1);
    const int n = (rv1 - rv0) * W * C8in;
    const uint16_t* src = a.in + a.in_vs * v + ((size_t)job_image(j) * H + rv0) * W * Cin;
#pragma unroll
    for (int q = 0; q < kPwDwPieces; ++q) {
      const int p = threadIdx.x + 256 * q;
      if (p < n) pre[q] = *reinterpret_cast<const cnn_u32x4*>(src + (size_t)p * 8);
    }
  };
  auto commit = [&](int j) {
    int rv0, rv1;
    strip_rows(job_row(j), rv0, rv1);
    const int n = (rv1 - rv0) * W * C8in;
#pragma unroll
    for (int q = 0; q < kPwDwPieces; ++q) {
      const int p = threadIdx.x + 256 * q;
      if (p < n) {
        const int px = (int)__umulhi((uint32_t)p, a.c8in_magic);   // p / C8in
        *reinterpret_cast<cnn_u32x4*>(al + (size_t)px * AS + (p - px * C8in) * 8) = pre[q];
      }
    }
  };
  // this wave's NT channel tiles (wave, wave + 4; Cout = 128 NT): weights as
  // bf16 A operands and the biases of the accumulator rows, loaded once
  cnn_u32x4 awt[NT][8];
  float biast[NT][16];
#pragma unroll
  for (int u = 0; u < NT; ++u) {
    const int n0 = min(wave + 4 * u, Cout / 32 - 1) * 32;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      if (s < KS) {
        const int k = 16 * s + 8 * lh;
        const float* src = Wv + ((size_t)(k / 32) * Cout + n0 + l32) * 32 + k % 32;
        const float4 w0 = *reinterpret_cast<const float4*>(src);
        const float4 w1 = *reinterpret_cast<const float4*>(src + 4);
        awt[u][s] = cnn_u32x4{f32_to_bf16_bits(w0.x) | (uint32_t)f32_to_bf16_bits(w0.y) << 16,
                              f32_to_bf16_bits(w0.z) | (uint32_t)f32_to_bf16_bits(w0.w) << 16,
                              f32_to_bf16_bits(w1.x) | (uint32_t)f32_to_bf16_bits(w1.y) << 16,
                              f32_to_bf16_bits(w1.z) | (uint32_t)f32_to_bf16_bits(w1.w) << 16};
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) biast[u][r] = pb[n0 + crow(r, lane)];
  }
  fetch(0);
  commit(0);
  __syncthreads();
  for (int j = 0; j < njobs; ++j) {
    const bool more = j + 1 < njobs;
    if (more) fetch(j + 1);                                  // in flight through this strip's work
    const int yo0 = job_row(j);
    uint16_t* ov = a.out + a.out_vs * v + (size_t)job_image(j) * a.Ho * a.Wo * Cout;
    const int rbase = S * yo0 - 1;
    int rv0, rv1;
    strip_rows(yo0, rv0, rv1);
    const int M = (rv1 - rv0) * W, mt = (M + 31) / 32;
#pragma unroll
    for (int u = 0; u < NT; ++u) {
      const int nt = wave + 4 * u;
      const int n0 = nt * 32;
      const cnn_u32x4* aw = awt[u];
      const float* bias = biast[u];
      for (int m = 0; m < mt; ++m) {
        const int pm = min(m * 32 + l32, M - 1);            // pixels past the strip: computed, never stored
        const uint16_t* ap = al + (size_t)pm * AS + 8 * lh;
        f32x16_t acc = zero16();
#pragma unroll
        for (int s = 0; s < 8; ++s)
          if (s < KS) acc = cnn_mma(aw[s], *reinterpret_cast<const cnn_u32x4*>(ap + 16 * s), acc);
        float f[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float z = acc[r] + bias[r];
          f[r] = z > 0.0f ? z : 0.0f;
        }
        uint32_t pk[8];
        to_bf16x2(f, pk);                                    // pk[i]: channels crow(2i), crow(2i) + 1
        if (m * 32 + l32 < M) {
          uint16_t* dst = pl + ((size_t)(rv0 - rbase) * W + m * 32 + l32) * PS + n0 + 4 * lh;
#pragma unroll
          for (int q = 0; q < 4; ++q) *reinterpret_cast<uint2*>(dst + 8 * q) = make_uint2(pk[2 * q], pk[2 * q + 1]);
        }
      }
    }
    __syncthreads();                                         // pointwise strip complete; its inputs are free
    if (more) commit(j + 1);                                 // before this strip's stores join the wait
    // depthwise items (output pixel, 8 channels): a thread keeps its channels
    // (256 is a multiple of Cout / 8) and steps through the strip's pixels
    constexpr int C8 = 16 * NT;
    const int R = min(a.R, a.Ho - yo0), npix = R * a.Wo;
    const int c0 = (threadIdx.x % C8) * 8;
    for (int pix = threadIdx.x / C8; pix < npix; pix += 256 / C8) {
      const int yr = (int)__umulhi((uint32_t)pix, a.wo_magic);     // pix / Wo
      const int xo = pix - yr * a.Wo, yo = yo0 + yr;
      auto tap = [&](int t) {
        const int r = S * yo + t / 3 - 1, xx = S * xo + t % 3 - 1;
        const bool in = r >= 0 && r < H && xx >= 0 && xx < W;
        return in ? *reinterpret_cast<const uint4*>(pl + ((size_t)(r - rbase) * W + xx) * PS + c0)
                  : make_uint4(0, 0, 0, 0);
      };
      float acc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
      cnn_dw_dot(tap, dt + c0, Cout, acc);
      float f[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float z = acc[j] + dbias[c0 + j];
        f[j] = z > 0.0f ? z : 0.0f;
      }
      uint32_t pk[4];
      to_bf16x2(f, pk);
      *reinterpret_cast<uint4*>(ov + ((size_t)yo * a.Wo + xo) * Cout + c0) = make_uint4(pk[0], pk[1], pk[2], pk[3]);
    }
    __syncthreads();                                         // next inputs staged; this strip's outputs read
  }
}

// global average pooling: one thread per pooled row (image) and 8 channels
__global__ __launch_bounds__(256) void k_cnn_pool(CnnPoolArgs a) {
  const int v = blockIdx.y, C8 = a.C / 8;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= kCnnChunk * C8) return;
  const int row = i / C8, c0 = (i % C8) * 8;
  float f[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = 0.0f;
  const uint16_t* src = a.in + a.in_vs * v + (size_t)row * a.HW * a.C + c0;
  for (int p = 0; p < a.HW; ++p) {
    const uint4 q = *reinterpret_cast<const uint4*>(src + (size_t)p * a.C);
    const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] += bf16_bits_to_f32((uint16_t)(w4[j >> 1] >> (16 * (j & 1))));
  }
  const float inv = 1.0f / (float)a.HW;
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] *= inv;
  uint32_t pk[4];
  to_bf16x2(f, pk);
  *reinterpret_cast<uint4*>(a.out + a.out_vs * v + (size_t)row * a.C + c0) = make_uint4(pk[0], pk[1], pk[2], pk[3]);
}

namespace {

int round_up32(int x) { return (x + 31) / 32 * 32; }

// ceil(2^32 / d): for n, d < 2^16, (n * m) >> 32 is exactly n / d
uint32_t cnn_magic(int d) { return (uint32_t)((((uint64_t)1 << 32) + (uint64_t)d - 1) / (uint64_t)d); }

// LDS bytes of the stem's zero-padded bf16 image
size_t cnn_stem_lds(int H, int W, int C) { return ((size_t)(H + 2) * (W + 2) * C * 2 + 15) / 16 * 16; }

// LDS bytes of the fused pointwise + depthwise kernel for strips of R output
// rows: the pointwise inputs (S (R - 1) + 3 rows of W pixels x (Cin + 8) bf16),
// the pointwise outputs (the same rows x (Cout + 8) bf16), the depthwise tap
// pairs and biases
size_t cnn_pwdw_lds(int S, int R, int W, int Cin, int Cout) {
  const size_t px = (size_t)(S * (R - 1) + 3) * W;
  return ((px * (Cin + 8) + 7) & ~(size_t)7) * 2 + ((px * (Cout + 8) + 7) & ~(size_t)7) * 2 + (size_t)6 * Cout * 4;
}

// Strip rows of the fused kernel for pointwise Cin -> Cout on H x W followed
// by a depthwise stride S to Ho rows: the most rows whose LDS fits 64 KiB and
// whose inputs fit the staging registers, or 0 when the pair runs unfused.
int cnn_fuse_rows(int Cin, int Cout, int W, int S, int Ho) {
  if (Cin % 32 || Cin > 128 || (Cout != 128 && Cout != 256)) return 0;
  int R = 0;
  for (int r = 1; r <= Ho; ++r) {
    const size_t pieces = (size_t)(S * (r - 1) + 3) * W * Cin / 8;
    if (cnn_pwdw_lds(S, r, W, Cin, Cout) <= 64 * 1024 && pieces <= (size_t)kPwDwPieces * 256) R = r;
  }
  return R;
}

// word `word` of the Philox4x32-10 block at counter (c0, c1, c2, stream), key seed
uint32_t draw_word(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t stream, uint32_t word) {
  const uint32_t ctr[4] = {c0, c1, c2, stream};
  const uint32_t key[2] = {(uint32_t)(seed & 0xffffffffu), (uint32_t)(seed >> 32)};
  uint32_t out[4];
  philox4x32_10_host(ctr, key, out);
  return out[word];
}
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct CnnTensor {
  int K = 0, N = 0, Kp = 0, Np = 0;
  size_t Wm = 0, bias = 0, mask = 0, base_w = 0, base_b = 0;
  size_t pack = 0;                            // prediction copy: [P][K][N] fp32 (stem), [P][5][N] tap pairs (depthwise)
  bool packed = false, pairs = false;
};

struct CnnLayout {
  int P = 0, nb = 0, H = 0, W = 0, C = 0, classes = 0, n_chunks = 0;
  int64_t n_test = 0;
  int stem = 0, ch[GEVO_CNN_MAX_BLOCKS] = {0}, stride[GEVO_CNN_MAX_BLOCKS] = {0};
  int fuse_R[GEVO_CNN_MAX_BLOCKS] = {0};      // > 0: pointwise i runs fused with depthwise i + 1, R rows per strip
  int hin[GEVO_CNN_MAX_BLOCKS + 1] = {0}, win[GEVO_CNN_MAX_BLOCKS + 1] = {0};   // spatial size entering block i (last: the head)
  int nt = 0;
  CnnTensor t[2 * GEVO_CNN_MAX_BLOCKS + 2];  // stem, (dw, pw) per block, fc
  size_t act_vs = 0;                          // elements per variant of an activation buffer
  size_t thresh = 0, aux = 0, actA = 0, actB = 0, pooled = 0, labels = 0, part_ce = 0, part_corr = 0;
  size_t test_ce = 0, test_corr = 0, total = 0;
};

gevo_status cnn_layout(const gevo_cnn_config* c, int64_t n_test, CnnLayout& y) {
  if (!c || c->abi_version != GEVO_ABI_VERSION) return GEVO_E_ARG;
  if (c->P < 1 || c->height < 1 || c->width < 1 || c->channels < 1 || n_test < 1) return GEVO_E_ARG;
  if (c->n_blocks < 1 || c->n_blocks > GEVO_CNN_MAX_BLOCKS) return GEVO_E_UNSUPPORTED;
  if (c->channels > 4 || c->stem_channels % 32 || c->stem_channels == 0 || c->stem_channels > 512)
    return GEVO_E_UNSUPPORTED;
  if (c->classes < 2 || c->classes > 32) return GEVO_E_UNSUPPORTED;
  if (c->height > 1024 || c->width > 1024 || c->P > 65535) return GEVO_E_UNSUPPORTED;
  if (!(c->dens_lo >= 0.0f && c->dens_hi <= 1.0f && c->dens_lo <= c->dens_hi)) return GEVO_E_ARG;
  if (!(c->noise_rel_std >= 0.0f)) return GEVO_E_ARG;
  y.P = (int)c->P; y.nb = (int)c->n_blocks; y.H = (int)c->height; y.W = (int)c->width; y.C = (int)c->channels;
  y.classes = (int)c->classes; y.n_test = n_test; y.stem = (int)c->stem_channels;
  y.n_chunks = (int)((n_test + kCnnChunk - 1) / kCnnChunk);
  int h = y.H, w = y.W, ch = y.stem;
  size_t act = (size_t)kCnnChunk * h * w * ch;
  y.nt = 0;
  auto add = [&](int K, int N, int Np) {
    CnnTensor& t = y.t[y.nt++];
    t.K = K; t.N = N; t.Kp = round_up32(K); t.Np = Np;
  };
  add(9 * y.C, y.stem, y.stem);
  y.t[0].packed = true;
  for (int i = 0; i < y.nb; ++i) {
    const int s = (int)c->block_stride[i], co = (int)c->block_channels[i];
    if ((s != 1 && s != 2) || co % 128 || co == 0 || co > 1024) return GEVO_E_UNSUPPORTED;
    y.hin[i] = h; y.win[i] = w; y.stride[i] = s; y.ch[i] = co;
    h = (h - 1) / s + 1;
    w = (w - 1) / s + 1;
    if (((size_t)kCnnChunk * h * w) % 256) return GEVO_E_UNSUPPORTED;   // pointwise GEMM rows
    add(9, ch, ch);                                   // depthwise taps of each channel
    y.t[y.nt - 1].packed = true;
    y.t[y.nt - 1].pairs = true;
    add(ch, co, co);                                  // pointwise
    act = std::max(act, (size_t)kCnnChunk * h * w * std::max(ch, co));
    ch = co;
  }
  y.hin[y.nb] = h; y.win[y.nb] = w;
  {
    int cin = y.stem;
    for (int i = 0; i + 1 < y.nb; ++i) {
      y.fuse_R[i] = cnn_fuse_rows(cin, y.ch[i], y.win[i + 1], y.stride[i + 1], y.hin[i + 2]);
      cin = y.ch[i];
    }
  }
  if (cnn_stem_lds(y.H, y.W, y.C) > 56 * 1024) return GEVO_E_UNSUPPORTED;   // the stem stages one image in LDS
  add(ch, y.classes, 32);                             // head, in the output kernel's 32-class layout
  y.act_vs = act;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off = align256(off + bytes); return at; };
  const size_t P = (size_t)y.P;
  for (int i = 0; i < y.nt; ++i) {
    CnnTensor& t = y.t[i];
    t.Wm = take(P * t.Np * t.Kp * 4);
    t.bias = take(P * t.Np * 4);
    t.mask = take(P * t.Np * (t.Kp / 32) * 4);
    t.base_w = take((size_t)t.Np * t.Kp * 4);
    t.base_b = take((size_t)t.Np * 4);
    if (t.packed) t.pack = take(P * (t.pairs ? 5 : t.K) * t.N * 4);
  }
  y.thresh = take(P * 4);
  y.aux = take(P * 4);                                // learning rates and bias bits the output kernel reads
  y.actA = take(P * y.act_vs * 2);
  y.actB = take(P * y.act_vs * 2);
  y.pooled = take(P * kCnnChunk * ch * 2);
  y.labels = take((size_t)y.n_chunks * kCnnChunk * 4);
  y.part_ce = take(P * y.n_chunks * 8);
  y.part_corr = take(P * y.n_chunks * 4);
  y.test_ce = take(P * 8);
  y.test_corr = take(P * 8);
  y.total = off;
  return GEVO_OK;
}

template <typename T>
T* at(char* ws, size_t off) { return reinterpret_cast<T*>(ws + off); }

}  // namespace

}  // namespace gevo

using namespace gevo;

struct gevo_cnn {
  gevo_cnn_config cfg{};
  CnnLayout y;
  char* ws = nullptr;
  hipStream_t stream = nullptr;
  const float* teX = nullptr;
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  bool predicted = false, timing_pending = false;
  double last_s = 0.0;
  std::vector<float> dens;
  // kernel-level timing (gevo_cnn_set_profiling)
  bool prof_on = false;
  struct ProfRec { int kind; hipEvent_t a, b; };
  std::vector<ProfRec> prof_pending;
  std::vector<hipEvent_t> ev_free, ev_all;
  double prof_ms[GEVO_CNN_KERNEL_KINDS] = {0};
  uint64_t prof_n[GEVO_CNN_KERNEL_KINDS] = {0};
};

namespace {

constexpr size_t kCnnProfBatch = 8192;   // launches between resolutions of pending timings

hipError_t cnn_prof_resolve(gevo_cnn* h) {
  if (h->prof_pending.empty()) return hipSuccess;
  const hipError_t err = hipStreamSynchronize(h->stream);
  if (err != hipSuccess) return err;
  for (const auto& r : h->prof_pending) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      h->prof_ms[r.kind] += (double)ms;
      h->prof_n[r.kind] += 1;
    }
    h->ev_free.push_back(r.a);
    h->ev_free.push_back(r.b);
  }
  h->prof_pending.clear();
  return hipSuccess;
}

hipEvent_t cnn_take_event(gevo_cnn* h) {
  if (!h->ev_free.empty()) {
    hipEvent_t e = h->ev_free.back();
    h->ev_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  h->ev_all.push_back(e);
  return e;
}

// events recorded by the dispatch of the next launch of this kind (none when profiling is off)
LaunchEv cnn_prof(gevo_cnn* h, int kind) {
  LaunchEv ev;
  if (!h->prof_on) return ev;
  if (h->prof_pending.size() >= kCnnProfBatch && cnn_prof_resolve(h) != hipSuccess) return ev;
  ev.start = cnn_take_event(h);
  ev.stop = cnn_take_event(h);
  if (!ev.start || !ev.stop) {
    if (ev.start) h->ev_free.push_back(ev.start);
    if (ev.stop) h->ev_free.push_back(ev.stop);
    return LaunchEv{};
  }
  h->prof_pending.push_back({kind, ev.start, ev.stop});
  return ev;
}

}  // namespace

#define CNN_HIP(x)                              \
  do {                                          \
    if ((x) != hipSuccess) return GEVO_E_HIP;   \
  } while (0)

extern "C" {

gevo_status gevo_cnn_param_count(const gevo_cnn_config* cfg, size_t* count) {
  if (!count) return GEVO_E_ARG;
  CnnLayout y;
  const gevo_status st = cnn_layout(cfg, 1, y);
  if (st != GEVO_OK) return st;
  size_t n = 0;
  for (int i = 0; i < y.nt; ++i) n += (size_t)y.t[i].K * y.t[i].N + y.t[i].N;
  *count = n;
  return GEVO_OK;
}

gevo_status gevo_cnn_workspace_bytes(const gevo_cnn_config* cfg, int64_t n_test, size_t* bytes) {
  if (!bytes) return GEVO_E_ARG;
  CnnLayout y;
  const gevo_status st = cnn_layout(cfg, n_test, y);
  if (st != GEVO_OK) return st;
  *bytes = y.total;
  return GEVO_OK;
}

gevo_status gevo_cnn_set_profiling(gevo_cnn* h, int enable) {
  if (!h) return GEVO_E_ARG;
  if (!enable && cnn_prof_resolve(h) != hipSuccess) return GEVO_E_HIP;
  h->prof_on = enable != 0;
  return GEVO_OK;
}

gevo_status gevo_cnn_kernel_stats(gevo_cnn* h, int kind, double* total_ms, uint64_t* launches) {
  if (!h || kind < 0 || kind >= GEVO_CNN_KERNEL_KINDS) return GEVO_E_ARG;
  if (cnn_prof_resolve(h) != hipSuccess) return GEVO_E_HIP;
  if (total_ms) *total_ms = h->prof_ms[kind];
  if (launches) *launches = h->prof_n[kind];
  return GEVO_OK;
}

void gevo_cnn_destroy(gevo_cnn* h) {
  if (!h) return;
  if (h->ev0) (void)hipEventDestroy(h->ev0);
  if (h->ev1) (void)hipEventDestroy(h->ev1);
  if (!h->ev_all.empty()) (void)hipStreamSynchronize(h->stream);
  for (hipEvent_t e : h->ev_all) (void)hipEventDestroy(e);
  delete h;
}

gevo_status gevo_cnn_init(const gevo_cnn_config* cfg, void* d_ws, size_t ws_bytes, const float* base_params,
                          const float* d_test_x, const int32_t* d_test_y, int64_t n_test, void* hip_stream,
                          gevo_cnn** out) {
  if (!out) return GEVO_E_ARG;
  *out = nullptr;
  CnnLayout y;
  gevo_status st = cnn_layout(cfg, n_test, y);
  if (st != GEVO_OK) return st;
  if (!d_ws || !base_params || !d_test_x || !d_test_y) return GEVO_E_ARG;
  if (ws_bytes < y.total || (reinterpret_cast<uintptr_t>(d_ws) & 255)) return GEVO_E_WORKSPACE;
  gevo_cnn* h = new (std::nothrow) gevo_cnn;
  if (!h) return GEVO_E_ARG;
  h->cfg = *cfg;
  h->y = y;
  h->ws = reinterpret_cast<char*>(d_ws);
  h->stream = reinterpret_cast<hipStream_t>(hip_stream);
  h->teX = d_test_x;
  auto fail = [&](gevo_status s) { gevo_cnn_destroy(h); return s; };
  if (hipEventCreate(&h->ev0) != hipSuccess || hipEventCreate(&h->ev1) != hipSuccess) return fail(GEVO_E_HIP);
  const int P = y.P;
  // per-variant density and mask threshold (host, fp64), drawn as for the
  // fully connected populations (stream kStreamDens)
  std::vector<uint32_t> thresh(P);
  std::vector<float> zeros(P, 0.0f);
  h->dens.resize(P);
  for (int v = 0; v < P; ++v) {
    const double u = (double)(draw_word(cfg->seed, 0, 0, (uint32_t)v, kStreamDens, 0) >> 8) * (1.0 / 16777216.0);
    const float rho = (float)((double)cfg->dens_lo + u * ((double)cfg->dens_hi - (double)cfg->dens_lo));
    h->dens[v] = rho;
    double t = floor((double)rho * 16777216.0 + 0.5);
    t = t < 0.0 ? 0.0 : (t > 16777216.0 ? 16777216.0 : t);
    thresh[v] = (uint32_t)t;
  }
  char* ws = h->ws;
  if (hipMemcpy(ws + y.thresh, thresh.data(), (size_t)P * 4, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(ws + y.aux, zeros.data(), (size_t)P * 4, hipMemcpyHostToDevice) != hipSuccess)
    return fail(GEVO_E_HIP);
  // base tensors, padded and transposed to [Np][Kp], then the variants
  size_t off = 0;
  for (int i = 0; i < y.nt; ++i) {
    const CnnTensor& t = y.t[i];
    std::vector<float> bw((size_t)t.Np * t.Kp, 0.0f), bb((size_t)t.Np, 0.0f);
    for (int k = 0; k < t.K; ++k)
      for (int n = 0; n < t.N; ++n) bw[(size_t)n * t.Kp + k] = base_params[off + (size_t)k * t.N + n];
    off += (size_t)t.K * t.N;
    for (int n = 0; n < t.N; ++n) bb[n] = base_params[off + n];
    off += (size_t)t.N;
    if (hipMemcpy(ws + t.base_w, bw.data(), bw.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(ws + t.base_b, bb.data(), bb.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
      return fail(GEVO_E_HIP);
    InitArgs a{};
    a.P = P; a.l_index = i; a.K = t.K; a.N = t.N; a.Kp = t.Kp; a.Np = t.Np;
    a.seed = cfg->seed;
    a.init_kind = 1;
    a.xavier_a = (float)sqrt(6.0 / ((double)t.K + (double)t.N));
    a.noise_std = cfg->noise_rel_std;
    a.base_w = at<const float>(ws, t.base_w);
    a.base_b = at<const float>(ws, t.base_b);
    a.thresh = at<const uint32_t>(ws, y.thresh);
    a.Wm = at<float>(ws, t.Wm);
    a.bias = at<float>(ws, t.bias);
    a.mask = at<uint32_t>(ws, t.mask);
    if (launch_init(a, h->stream, LaunchEv{}) != hipSuccess) return fail(GEVO_E_HIP);
    if (t.packed && t.pairs) {
      const int64_t n = (int64_t)P * 5 * t.N;
      hipLaunchKernelGGL(k_cnn_pack_pairs, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, h->stream,
                         at<const float>(ws, t.Wm), t.N, P, at<uint32_t>(ws, t.pack));
      if (hipGetLastError() != hipSuccess) return fail(GEVO_E_HIP);
    } else if (t.packed) {
      const int64_t n = (int64_t)P * t.K * t.N;
      hipLaunchKernelGGL(k_cnn_pack, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, h->stream,
                         at<const float>(ws, t.Wm), t.Kp, t.Np, t.K, t.N, P, at<float>(ws, t.pack));
      if (hipGetLastError() != hipSuccess) return fail(GEVO_E_HIP);
    }
  }
  // test labels per 64-image chunk, the last chunk's padding images marked -1
  std::vector<int32_t> ylab((size_t)n_test), tiles((size_t)y.n_chunks * kCnnChunk, -1);
  if (hipMemcpy(ylab.data(), d_test_y, (size_t)n_test * 4, hipMemcpyDeviceToHost) != hipSuccess) return fail(GEVO_E_HIP);
  for (int64_t r = 0; r < n_test; ++r) {
    if (ylab[r] < 0 || ylab[r] >= y.classes) return fail(GEVO_E_SHAPE);
    tiles[(size_t)r] = ylab[r];
  }
  if (hipMemcpy(ws + y.labels, tiles.data(), tiles.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
    return fail(GEVO_E_HIP);
  if (hipDeviceSynchronize() != hipSuccess) return fail(GEVO_E_HIP);
  *out = h;
  return GEVO_OK;
}

gevo_status gevo_cnn_predict(gevo_cnn* h) {
  if (!h) return GEVO_E_ARG;
  const CnnLayout& y = h->y;
  char* ws = h->ws;
  hipStream_t s = h->stream;
  const int P = y.P;
  CNN_HIP(hipEventRecord(h->ev0, s));
  for (int c = 0; c < y.n_chunks; ++c) {
    // stem: test images -> A
    const CnnTensor& ts = y.t[0];
    CnnStemArgs sa{};
    sa.x = h->teX; sa.n_test = y.n_test; sa.img0 = c * kCnnChunk;
    sa.H = y.H; sa.W = y.W; sa.Np = ts.Np;
    sa.w_magic = cnn_magic(y.W); sa.w2_magic = cnn_magic(y.W + 2);
    sa.wp = at<const float>(ws, ts.pack); sa.bias = at<const float>(ws, ts.bias);
    sa.out = at<uint16_t>(ws, y.actA); sa.out_vs = y.act_vs;
    LaunchEv ev = cnn_prof(h, GEVO_CNN_KERNEL_STEM);
    const dim3 sg(kCnnChunk, P);                                 // one workgroup per (variant, image)
    const size_t lds = cnn_stem_lds(y.H, y.W, y.C);
    switch (y.C) {
      case 1: hipExtLaunchKernelGGL(k_cnn_stem<1>, sg, dim3(256), lds, s, ev.start, ev.stop, 0, sa); break;
      case 2: hipExtLaunchKernelGGL(k_cnn_stem<2>, sg, dim3(256), lds, s, ev.start, ev.stop, 0, sa); break;
      case 3: hipExtLaunchKernelGGL(k_cnn_stem<3>, sg, dim3(256), lds, s, ev.start, ev.stop, 0, sa); break;
      default: hipExtLaunchKernelGGL(k_cnn_stem<4>, sg, dim3(256), lds, s, ev.start, ev.stop, 0, sa); break;
    }
    CNN_HIP(hipGetLastError());
    // activations ping-pong between the two buffers; `cur` holds the latest map
    uint16_t* cur = at<uint16_t>(ws, y.actA);
    uint16_t* other = at<uint16_t>(ws, y.actB);
    auto depthwise = [&](int i, int C) -> hipError_t {      // depthwise of block i: cur -> other
      const CnnTensor& td = y.t[1 + 2 * i];
      CnnDwArgs da{};
      da.in = cur; da.in_vs = y.act_vs;
      da.out = other; da.out_vs = y.act_vs;
      da.H = y.hin[i]; da.W = y.win[i]; da.C = C; da.Ho = y.hin[i + 1]; da.Wo = y.win[i + 1]; da.stride = y.stride[i];
      da.wp = at<const uint32_t>(ws, td.pack); da.bias = at<const float>(ws, td.bias);
      const int dw_threads = kCnnChunk * da.Wo * (C / 8);        // (image, column, 8 channels)
      const LaunchEv e = cnn_prof(h, GEVO_CNN_KERNEL_DEPTHWISE);
      const dim3 dg((dw_threads + 255) / 256, P);
      if (da.stride == 1)
        hipExtLaunchKernelGGL(k_cnn_dw<1>, dg, dim3(256), (size_t)6 * C * 4, s, e.start, e.stop, 0, da);
      else
        hipExtLaunchKernelGGL(k_cnn_dw<2>, dg, dim3(256), (size_t)6 * C * 4, s, e.start, e.stop, 0, da);
      std::swap(cur, other);
      return hipGetLastError();
    };
    CNN_HIP(depthwise(0, y.stem));
    int ch = y.stem;
    for (int i = 0; i < y.nb; ++i) {
      const CnnTensor& tp = y.t[2 + 2 * i];
      const int Hp = y.hin[i + 1], Wp = y.win[i + 1];          // the pointwise layer's spatial size
      if (i + 1 < y.nb && y.fuse_R[i] > 0) {
        // pointwise i and depthwise i + 1 in one kernel: cur -> other
        const CnnTensor& td = y.t[1 + 2 * (i + 1)];
        CnnPwDwArgs fa{};
        fa.in = cur; fa.in_vs = y.act_vs;
        fa.Wm = at<const float>(ws, tp.Wm); fa.pbias = at<const float>(ws, tp.bias);
        fa.dwp = at<const uint32_t>(ws, td.pack); fa.dbias = at<const float>(ws, td.bias);
        fa.out = other; fa.out_vs = y.act_vs;
        fa.H = Hp; fa.W = Wp; fa.Cin = ch; fa.Cout = y.ch[i];
        fa.Ho = y.hin[i + 2]; fa.Wo = y.win[i + 2]; fa.R = y.fuse_R[i];
        fa.ipw = Hp * Wp >= 1024 ? 1 : (Hp * Wp >= 256 ? 4 : 8);   // images per workgroup
        fa.wo_magic = cnn_magic(fa.Wo);
        fa.c8in_magic = cnn_magic(fa.Cin / 8);
        const int S = y.stride[i + 1];
        const size_t lds = cnn_pwdw_lds(S, fa.R, fa.W, fa.Cin, fa.Cout);
        const LaunchEv e = cnn_prof(h, GEVO_CNN_KERNEL_POINTWISE_DEPTHWISE);
        const dim3 fg(kCnnChunk / fa.ipw, P);
        if (S == 1 && fa.Cout == 128)
          hipExtLaunchKernelGGL((k_cnn_pwdw<1, 1>), fg, dim3(256), lds, s, e.start, e.stop, 0, fa);
        else if (S == 1)
          hipExtLaunchKernelGGL((k_cnn_pwdw<1, 2>), fg, dim3(256), lds, s, e.start, e.stop, 0, fa);
        else if (fa.Cout == 128)
          hipExtLaunchKernelGGL((k_cnn_pwdw<2, 1>), fg, dim3(256), lds, s, e.start, e.stop, 0, fa);
        else
          hipExtLaunchKernelGGL((k_cnn_pwdw<2, 2>), fg, dim3(256), lds, s, e.start, e.stop, 0, fa);
        CNN_HIP(hipGetLastError());
        std::swap(cur, other);                                     // cur: depthwise i + 1 output
        ch = y.ch[i];
      } else {
        FwdGemmArgs g{};
        g.A = cur; g.a_vs = y.act_vs;
        g.Wm = at<const float>(ws, tp.Wm); g.bias = at<const float>(ws, tp.bias);
        g.O = other; g.o_vs = y.act_vs;
        g.Kp = tp.Kp; g.Np = tp.Np; g.R = kCnnChunk * Hp * Wp; g.P = P;
        if (!fwd_gemm_supported(g.Kp, g.Np, g.R)) return GEVO_E_SHAPE;
        CNN_HIP(launch_fwd_gemm(g, s, cnn_prof(h, GEVO_CNN_KERNEL_POINTWISE)));
        std::swap(cur, other);
        ch = y.ch[i];
        if (i + 1 < y.nb) CNN_HIP(depthwise(i + 1, ch));
      }
    }
    CnnPoolArgs pa{};
    pa.in = cur; pa.in_vs = y.act_vs;
    pa.HW = y.hin[y.nb] * y.win[y.nb]; pa.C = ch;
    pa.out = at<uint16_t>(ws, y.pooled); pa.out_vs = (size_t)kCnnChunk * ch;
    ev = cnn_prof(h, GEVO_CNN_KERNEL_POOL);
    hipExtLaunchKernelGGL(k_cnn_pool, dim3((kCnnChunk * (ch / 8) + 255) / 256, P), dim3(256), 0, s, ev.start, ev.stop,
                          0, pa);
    CNN_HIP(hipGetLastError());
    const CnnTensor& tf = y.t[y.nt - 1];
    OutArgs<uint16_t> o{};
    o.Kp = tf.Kp; o.C = y.classes; o.Bp = kOutRows;
    o.Wm = at<float>(ws, tf.Wm); o.bias = at<float>(ws, tf.bias); o.mask = at<const uint32_t>(ws, tf.mask);
    o.bmask = at<const uint32_t>(ws, y.aux); o.lr = at<const float>(ws, y.aux);
    o.train = 0;
    o.Arows = at<const uint16_t>(ws, y.pooled); o.ar_vs = (size_t)kCnnChunk * ch;
    o.labels = at<const int32_t>(ws, y.labels) + (size_t)c * kCnnChunk;
    o.rows = kCnnChunk;                                          // padding images of the last chunk carry label -1
    o.chunk0 = c;
    o.n_chunks_total = y.n_chunks;
    o.part_ce = at<double>(ws, y.part_ce);
    o.part_correct = at<unsigned int>(ws, y.part_corr);
    CNN_HIP(launch_out<uint16_t>(o, P, s, cnn_prof(h, GEVO_CNN_KERNEL_HEAD)));
  }
  CNN_HIP(launch_reduce_partials(at<double>(ws, y.part_ce), at<unsigned int>(ws, y.part_corr), P, y.n_chunks,
                                 at<double>(ws, y.test_ce), at<unsigned long long>(ws, y.test_corr), s,
                                 cnn_prof(h, GEVO_CNN_KERNEL_REDUCE)));
  CNN_HIP(hipEventRecord(h->ev1, s));
  h->timing_pending = true;
  h->predicted = true;
  return GEVO_OK;
}

gevo_status gevo_cnn_scores(gevo_cnn* h, float* test_loss, float* test_acc, float* time_s) {
  if (!h) return GEVO_E_ARG;
  if (!h->predicted) return GEVO_E_ORDER;
  CNN_HIP(hipStreamSynchronize(h->stream));
  if (h->timing_pending) {
    float ms = 0.0f;
    CNN_HIP(hipEventElapsedTime(&ms, h->ev0, h->ev1));
    h->last_s = (double)ms * 1e-3;
    h->timing_pending = false;
  }
  const int P = h->y.P;
  std::vector<double> ce(P);
  std::vector<unsigned long long> corr(P);
  CNN_HIP(hipMemcpy(ce.data(), h->ws + h->y.test_ce, (size_t)P * 8, hipMemcpyDeviceToHost));
  CNN_HIP(hipMemcpy(corr.data(), h->ws + h->y.test_corr, (size_t)P * 8, hipMemcpyDeviceToHost));
  for (int v = 0; v < P; ++v) {
    if (test_loss) test_loss[v] = (float)(ce[v] / (double)h->y.n_test);
    if (test_acc) test_acc[v] = (float)((double)corr[v] / (double)h->y.n_test);
    if (time_s) time_s[v] = (float)(h->last_s / P);
  }
  return GEVO_OK;
}

gevo_status gevo_cnn_remove_layer(gevo_cnn* h, uint32_t v, uint32_t layer) {
  if (!h) return GEVO_E_ARG;
  const CnnLayout& y = h->y;
  if (v >= (uint32_t)y.P || layer >= (uint32_t)y.nt) return GEVO_E_ARG;
  if (layer == 0 || layer + 1 == (uint32_t)y.nt) return GEVO_E_UNSUPPORTED;   // the stem and the head stay
  const CnnTensor& t = y.t[layer];
  const bool depthwise = layer % 2 == 1;                                      // stem, (dw, pw) per block, head
  char* ws = h->ws;
  hipLaunchKernelGGL(k_cnn_identity, dim3(std::max(1, std::min(256, (t.Kp * t.Np + 255) / 256))), dim3(256), 0,
                     h->stream, at<float>(ws, t.Wm) + (size_t)v * t.Np * t.Kp, at<float>(ws, t.bias) + (size_t)v * t.Np,
                     at<uint32_t>(ws, t.mask) + (size_t)v * t.Np * (t.Kp / 32), t.Kp, t.Np, t.K, t.N,
                     depthwise ? 4 : -1);
  CNN_HIP(hipGetLastError());
  if (t.packed && t.pairs) {                                                  // the prediction copy of the taps
    const int64_t n = (int64_t)y.P * 5 * t.N;
    hipLaunchKernelGGL(k_cnn_pack_pairs, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, h->stream,
                       at<const float>(ws, t.Wm), t.N, y.P, at<uint32_t>(ws, t.pack));
    CNN_HIP(hipGetLastError());
  }
  return GEVO_OK;
}

gevo_status gevo_cnn_export(gevo_cnn* h, uint32_t v, float* params_out, uint8_t* mask_out, float* density_out) {
  if (!h) return GEVO_E_ARG;
  const CnnLayout& y = h->y;
  if (v >= (uint32_t)y.P) return GEVO_E_ARG;
  CNN_HIP(hipStreamSynchronize(h->stream));
  size_t off = 0, moff = 0;
  for (int i = 0; i < y.nt; ++i) {
    const CnnTensor& t = y.t[i];
    const size_t nw = (size_t)t.Np * t.Kp, words = (size_t)t.Np * (t.Kp / 32);
    std::vector<float> W(nw), b((size_t)t.Np);
    std::vector<uint32_t> M(words);
    CNN_HIP(hipMemcpy(W.data(), h->ws + t.Wm + (size_t)v * nw * 4, nw * 4, hipMemcpyDeviceToHost));
    CNN_HIP(hipMemcpy(b.data(), h->ws + t.bias + (size_t)v * t.Np * 4, (size_t)t.Np * 4, hipMemcpyDeviceToHost));
    CNN_HIP(hipMemcpy(M.data(), h->ws + t.mask + (size_t)v * words * 4, words * 4, hipMemcpyDeviceToHost));
    for (int k = 0; k < t.K; ++k)
      for (int n = 0; n < t.N; ++n) {
        if (params_out) params_out[off + (size_t)k * t.N + n] = W[((size_t)(k / 32) * t.Np + n) * 32 + k % 32];
        if (mask_out) mask_out[moff + (size_t)k * t.N + n] = (uint8_t)((M[(size_t)n * (t.Kp / 32) + k / 32] >> (k % 32)) & 1u);
      }
    off += (size_t)t.K * t.N;
    moff += (size_t)t.K * t.N;
    for (int n = 0; n < t.N; ++n)
      if (params_out) params_out[off + n] = b[n];
    off += (size_t)t.N;
  }
  if (density_out) *density_out = h->dens[v];
  return GEVO_OK;
}

}  // extern "C"
