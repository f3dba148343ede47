// conv_bf16.hip -- 3x3 / stride 1 / pad 1 convolution forward and data
// gradient with bf16 operands on the bf16 MFMA (v_mfma_f32_32x32x16_bf16,
// fp32 accumulation), for SB_BF16 tensors.
//
// The same implicit GEMM as the fp32 kernels (rows = output channels,
// columns = output pixels, reduction = input channels x 9 taps, the input
// halo of a 16-channel chunk staged once in LDS and read at 9 shifted
// windows).  A block owns 64 output channels x 256 output pixels; each of
// its four waves owns all 64 channels x 64 pixels (2 x 2 tiles of 32 x 32).
// A lane of this MFMA supplies 8 consecutive reduction values (8
// consecutive input channels at one tap), so both operands sit in LDS as
// planes of 8 channels, each 16-byte row one (pixel or output channel):
//   * filters, packed per (output-channel tile, chunk) as
//     [tap][ci / 8][co][ci % 8] (filter_pack, PackCI8), staged as is;
//   * input halo as [ci / 8][halo pixel][ci % 8], transposed from NCHW on
//     its way in: a lane loads V consecutive columns of one channel (V = 8,
//     4, 2 when the width allows, else 1) and stores them as V 2-byte
//     writes 16 bytes apart.
// The 32 lanes of an operand read fetch 32 consecutive 16-byte rows, so the
// reads are free of bank conflicts without padding.
//
// The data gradient is the same contraction with the filters transposed and
// rotated (done by the pack).  Splits over channel chunks, the epilogue and
// the split reduction are the fp32 path's.
#include "conv_common.hpp"

#include <algorithm>
#include <cstdio>
#include <mutex>

namespace sb {

typedef short s8 __attribute__((ext_vector_type(8)));
typedef float f16 __attribute__((ext_vector_type(16)));

// D(32x32) += A(32x16) * B(16x32), bf16 in / fp32 accumulate.  Lane l
// supplies A[l%32][8*(l/32) + j] and B[8*(l/32) + j][l%32] (j = 0..7) and
// receives D[8*(v/4) + 4*(l/32) + v%4][l%32] in element v.
__device__ __forceinline__ f16 mfma32x32x16bf16(s8 a, s8 b, f16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <int TH_, int TW_, int IMGS_, int NB_ = 2>
struct BTile {
  static constexpr int TH = TH_, TW = TW_, IMGS = IMGS_;
  static constexpr int BM = IMGS * TH * TW;
  static_assert(BM == 256 || BM == 512, "pixel tile must hold 256 or 512 pixels");
  static constexpr int WP = BM / 4;                 // pixels per wave
  static constexpr int MB = WP / 32;                // 32-pixel MFMA blocks per wave
  static constexpr int NB = NB_;                    // 32-channel MFMA blocks per wave
  static constexpr int BN = 32 * NB, CK = 16;
  static constexpr int HH = TH + 2, HW = TW + 2;
  static constexpr int ROWS = IMGS * HH;            // halo rows
  static constexpr int PLANE = ROWS * HW;           // halo pixels
  static constexpr int WTS = 9 * BN * CK;           // filter elements per chunk
  static constexpr int WTS_V = WTS / 8;             // 16-byte rows of filters
  static constexpr int WTS_I = (WTS_V + 255) / 256;
  static constexpr int LDS_X = 2 * PLANE * 8;       // bf16 elements
  static constexpr int LDS_BUF = LDS_X + WTS;
  static_assert(LDS_X % 8 == 0 && LDS_BUF % 8 == 0, "16-byte aligned regions");
  static constexpr size_t LDS_BYTES = 2 * LDS_BUF * sizeof(u16);
  static_assert(LDS_BYTES <= 80 * 1024, "two blocks must fit in the 160 KB of LDS");
  // Pixel p of the tile: images outermost, then rows, then columns; a wave
  // owns WP consecutive pixels (MB blocks of 32).
  __host__ __device__ static constexpr int img_of(int p) { return p / (TH * TW); }
  __host__ __device__ static constexpr int yy_of(int p) { return p % (TH * TW) / TW; }
  __host__ __device__ static constexpr int xx_of(int p) { return p % TW; }
  // Halo pixel of (image, halo row, halo column).
  __host__ __device__ static constexpr int hp(int img, int hy, int hx) {
    return (img * HH + hy) * HW + hx;
  }
};

// ONE: a single LDS buffer (for short channel loops: a block then needs
// about half the LDS, so more blocks share a CU and one block's prologue and
// epilogue overlap another's MFMAs); the next chunk still loads into
// registers while the current one is computed.
template <class T>
__host__ __device__ constexpr size_t one_buf_lds_bytes() {
  return (T::LDS_BUF > T::BN * (T::BM + 8) ? T::LDS_BUF : T::BN * (T::BM + 8)) * sizeof(u16);
}

template <class T, bool DGRAD, int V, bool ONE = false>
__global__ __launch_bounds__(256, 2) void conv3x3_igemm_bf16(ConvArgs a) {
  extern __shared__ u16 ldsb[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lc = lane & 31, lh = lane >> 5;

  int bt = blockIdx.x;
  const int tx = bt % a.tiles_w; bt /= a.tiles_w;
  const int ty = bt % a.tiles_h;
  const int tn = bt / a.tiles_h;
  const int n0 = tn * T::IMGS, h0 = ty * T::TH, w0 = tx * T::TW;
  const int co0 = blockIdx.y * T::BN;
  const int kc0 = blockIdx.z * a.chunks_per_split;
  const int kc1 = min(a.nchunks, kc0 + a.chunks_per_split);
  const int HWs = a.H * a.W;

  // Halo staging.  Thread -> channel ci = tid % 16 and a set of (row,
  // column piece) combinations u = tid / 16 + 16 * round, rows fastest.
  // Interior pieces cover tile columns vi*V .. vi*V+V-1 (halo columns + 1);
  // the edge columns (halo columns 0 and TW+1) are single loads.
  constexpr int VPR = T::TW / V;                    // pieces per row
  constexpr int XI = (T::ROWS * VPR + 15) / 16;
  constexpr int EI = (T::ROWS * 2 + 15) / 16;
  const int ci = tid & 15;
  int x_off[XI], x_lds[XI], e_off[EI], e_lds[EI];
#pragma unroll
  for (int i = 0; i < XI; ++i) {
    const int u = (tid >> 4) + 16 * i;
    const int row = u % T::ROWS, vi = u / T::ROWS;
    const int img = row / T::HH, hy = row % T::HH;
    const int h = h0 + hy - 1, w = w0 + vi * V;
    const bool ok = u < T::ROWS * VPR && n0 + img < a.N && (unsigned)h < (unsigned)a.H &&
                    w < a.W;
    x_off[i] = ok ? (img * a.Cin + ci) * HWs + h * a.W + w : -1;   // from image n0
    x_lds[i] = u < T::ROWS * VPR ? ((ci >> 3) * T::PLANE + T::hp(img, hy, 1 + vi * V)) * 8 + (ci & 7)
                                 : -1;
  }
#pragma unroll
  for (int i = 0; i < EI; ++i) {
    const int u = (tid >> 4) + 16 * i;
    const int row = u % T::ROWS, side = u / T::ROWS;
    const int img = row / T::HH, hy = row % T::HH;
    const int h = h0 + hy - 1, w = side ? w0 + T::TW : w0 - 1;
    const bool ok = u < T::ROWS * 2 && n0 + img < a.N && (unsigned)h < (unsigned)a.H &&
                    (unsigned)w < (unsigned)a.W;
    e_off[i] = ok ? (img * a.Cin + ci) * HWs + h * a.W + w : -1;
    e_lds[i] = u < T::ROWS * 2
                   ? ((ci >> 3) * T::PLANE + T::hp(img, hy, side ? T::TW + 1 : 0)) * 8 + (ci & 7)
                   : -1;
  }
  // Operand rows of this lane: pixel lc of each of the wave's two pixel
  // blocks (halo pixel at tap (0, 0)), channel-plane lh.
  int b_off[T::MB];
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb) {
    const int p = wave * T::WP + mb * 32 + lc;
    b_off[mb] = (lh * T::PLANE + T::hp(T::img_of(p), T::yy_of(p), T::xx_of(p))) * 8;
  }

  f16 acc[T::NB][T::MB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i)
#pragma unroll
    for (int j = 0; j < T::MB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const rsrc_t xr = input_rsrc<u16>(a, n0, T::IMGS);
  const rsrc_t wr = packed_rsrc<u16, T::WTS>(a, blockIdx.y);
  typedef typename std::conditional<(V > 1), Vec<(V > 1 ? V : 2)>, u16>::type Piece;
  Piece rx[XI];
  u16 re[EI];
  s8 rw[T::WTS_I];
  auto gload = [&](int kc) {
    const int cb = kc * T::CK;
    const int cleft = a.Cin - cb - ci;               // this lane's channel valid if > 0
#pragma unroll
    for (int i = 0; i < XI; ++i) {
      const uint32_t off =
          x_off[i] >= 0 && cleft > 0 ? (uint32_t)(x_off[i] + cb * HWs) * 2u : kOOB;
      if constexpr (V > 1) rx[i] = load_vec<V>(xr, off);
      else rx[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(xr, (int)off, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < EI; ++i)
      re[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(
          xr, e_off[i] >= 0 && cleft > 0 ? (int)((uint32_t)(e_off[i] + cb * HWs) * 2u) : (int)kOOB,
          0, 0);
#pragma unroll
    for (int i = 0; i < T::WTS_I; ++i) {
      const int g = tid + 256 * i;
      const uint32_t off = g < T::WTS_V ? (uint32_t)(kc * T::WTS + g * 8) * 2u : kOOB;
      rw[i] = __builtin_bit_cast(s8, __builtin_amdgcn_raw_buffer_load_b128(wr, (int)off, 0, 0));
    }
  };
  auto lstore = [&](int buf) {
    u16* X = ldsb + buf * T::LDS_BUF;
    u16* Wl = X + T::LDS_X;
#pragma unroll
    for (int i = 0; i < XI; ++i) {
      if (x_lds[i] < 0) continue;
      u16* q = X + x_lds[i];
      if constexpr (V > 1) {
#pragma unroll
        for (int j = 0; j < V / 2; ++j) {
          q[(2 * j) * 8] = (u16)(rx[i].d[j] & 0xffffu);
          q[(2 * j + 1) * 8] = (u16)(rx[i].d[j] >> 16);
        }
      } else {
        q[0] = rx[i];
      }
    }
#pragma unroll
    for (int i = 0; i < EI; ++i)
      if (e_lds[i] >= 0) X[e_lds[i]] = re[i];
#pragma unroll
    for (int i = 0; i < T::WTS_I; ++i) {
      const int g = tid + 256 * i;
      if (g < T::WTS_V) *reinterpret_cast<s8*>(Wl + g * 8) = rw[i];
    }
  };
  auto compute = [&](int buf) {
    const u16* X = ldsb + buf * T::LDS_BUF;
    const u16* Wl = X + T::LDS_X;
    // The operands of tap t + 1 are read before tap t's MFMAs are issued,
    // so each read has a whole tap's MFMAs to arrive under.
    s8 fa[2][T::NB], fb[2][T::MB];
    auto rd = [&](int t, int s) {
      const int toff = T::hp(0, t / 3, t % 3) * 8;
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
        fa[s][nb] = *reinterpret_cast<const s8*>(Wl + ((t * 2 + lh) * T::BN + nb * 32 + lc) * 8);
#pragma unroll
      for (int mb = 0; mb < T::MB; ++mb)
        fb[s][mb] = *reinterpret_cast<const s8*>(X + b_off[mb] + toff);
    };
    rd(0, 0);
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      if (t + 1 < 9) rd(t + 1, (t + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);   // keep those reads ahead of the MFMAs
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb)
          acc[nb][mb] = mfma32x32x16bf16(fa[t & 1][nb], fb[t & 1][mb], acc[nb][mb]);
    }
  };

  const int nk = kc1 - kc0;
  if constexpr (ONE) {
    if (nk > 0) {
      gload(kc0);
      lstore(0);
    }
    __syncthreads();
    for (int t = 0; t < nk; ++t) {
      if (t + 1 < nk) gload(kc0 + t + 1);
      compute(0);
      __syncthreads();
      if (t + 1 < nk) {
        lstore(0);
        __syncthreads();
      }
    }
  } else {
    if (nk > 0) {
      gload(kc0);
      lstore(0);
      if (nk > 1) gload(kc0 + 1);
    }
    __syncthreads();
    for (int t = 0; t < nk; ++t) {
      const int buf = t & 1;
      if (t + 1 < nk) lstore(buf ^ 1);
      if (t + 2 < nk) gload(kc0 + t + 2);
      compute(buf);
      __syncthreads();
    }
  }

  // acc[nb][mb] element v: output channel co0 + nb*32 + 8*(v/4) + 4*lh +
  // v%4 of pixel wave*64 + mb*32 + lc.
  int pix[T::MB];                                    // offset from image n0, -1 outside
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb) {
    const int p = wave * T::WP + mb * 32 + lc;
    const int img = T::img_of(p), h = h0 + T::yy_of(p), w = w0 + T::xx_of(p);
    pix[mb] = n0 + img < a.N && h < a.H && w < a.W ? img * a.Cout * HWs + h * a.W + w : -1;
  }
  auto co_of = [&](int nb, int v) { return co0 + nb * 32 + 8 * (v >> 2) + 4 * lh + (v & 3); };
  if (a.splits > 1) {
    float* mine = a.part + (size_t)blockIdx.z * a.N * a.Cout * HWs + (size_t)n0 * a.Cout * HWs;
#pragma unroll
    for (int mb = 0; mb < T::MB; ++mb) {
      if (pix[mb] < 0) continue;
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int co = co_of(nb, v);
          if (co < a.Cout) mine[pix[mb] + co * HWs] = acc[nb][mb][v];
        }
    }
    return;
  }
  // The block's BN x BM outputs go through LDS ([channel][pixel], bias and
  // ReLU applied, rounded to bf16), then out to memory in pieces of V
  // consecutive pixels of one channel, the ReLU mask read in the same
  // pieces; every mask load is issued before the first store.
  constexpr int EP = T::BM + 8;                      // LDS row pitch (bf16)
  static_assert(T::BN * EP * sizeof(u16) <= (ONE ? one_buf_lds_bytes<T>() : T::LDS_BYTES),
                "output tile fits the staging LDS");
  u16* E = ldsb;
#pragma unroll
  for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int co = co_of(nb, v);
      const float bv = a.bias && co < a.Cout ? a.bias[co] : 0.f;
#pragma unroll
      for (int mb = 0; mb < T::MB; ++mb) {
        float r = acc[nb][mb][v] + bv;
        if (a.relu && !(r > 0.f)) r = 0.f;
        E[(co - co0) * EP + wave * T::WP + mb * 32 + lc] = f32_to_bf16(r);
      }
    }
  __syncthreads();
  constexpr int PPR = T::BM / V;                     // pieces per channel row
  constexpr int EPI = T::BN * PPR / 256;             // pieces per thread
  static_assert(T::BN * PPR % 256 == 0, "whole rounds of pieces");
  int goff[EPI];                                     // from image n0, -1 outside
#pragma unroll
  for (int i = 0; i < EPI; ++i) {
    const int q = tid + 256 * i;
    const int col = q / PPR, p = (q % PPR) * V;
    const int img = T::img_of(p), h = h0 + T::yy_of(p), w = w0 + T::xx_of(p);
    const int co = co0 + col;
    goff[i] = co < a.Cout && n0 + img < a.N && h < a.H && w < a.W
                  ? (img * a.Cout + co) * HWs + h * a.W + w : -1;
  }
  typedef typename std::conditional<(V > 1), Vec<(V > 1 ? V : 2)>, u16>::type Piece;
  Piece mk[EPI];
  if (a.mask) {
    const int cnt = min(T::IMGS, a.N - n0);
    const rsrc_t mr = make_rsrc((const u16*)a.mask + (size_t)n0 * a.Cout * HWs,
                                (uint32_t)((size_t)cnt * a.Cout * HWs * 2));
#pragma unroll
    for (int i = 0; i < EPI; ++i) {
      const uint32_t off = goff[i] >= 0 ? (uint32_t)goff[i] * 2u : kOOB;
      if constexpr (V > 1) mk[i] = load_vec<V>(mr, off);
      else mk[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(mr, (int)off, 0, 0);
    }
  }
  // A bf16 mask value m keeps the output iff m > 0: bits 0x0001..0x7f80.
  auto keep = [](uint32_t m16) { return ((m16 - 1u) & 0xffffu) < 0x7f80u; };
  u16* out = (u16*)a.out + (size_t)n0 * a.Cout * HWs;
#pragma unroll
  for (int i = 0; i < EPI; ++i) {
    if (goff[i] < 0) continue;
    const int q = tid + 256 * i;
    const u16* src = E + (q / PPR) * EP + (q % PPR) * V;
    if constexpr (V > 1) {
      Vec<V> o = lds_vec<V>(src);
#pragma unroll
      for (int j = 0; j < V / 2; ++j) {
        uint32_t d = o.d[j];
        if (a.mask) {
          const uint32_t m = mk[i].d[j];
          if (!keep(m & 0xffffu)) d &= 0xffff0000u;
          if (!keep(m >> 16)) d &= 0x0000ffffu;
        }
        o.d[j] = d;
      }
      store_vec<V>(out + goff[i], o);
    } else {
      u16 d = src[0];
      if (a.mask && !keep(mk[i])) d = 0;
      out[goff[i]] = d;
    }
  }
}

// ------------------------------------------------------ channel-blocked --
// The same contraction on channel-blocked tensors (SB_NCHW8C: element
// (n, c, h, w) at ((n * C/8 + c/8) * H + h) * W + w) * 8 + c % 8, C a
// multiple of 8).  Eight consecutive channels of a pixel are one 16-byte
// piece, which is exactly what an MFMA lane supplies, so the input halo is
// staged as whole pieces: one 16-byte load and one 16-byte LDS store per
// (channel block, halo pixel), no transposition.  The compute is the NCHW
// kernel's.  The output tile goes out through LDS as [pixel][channel] rows
// and leaves as 16-byte pieces (one pixel's 8 channels), the ReLU mask read
// in the same pieces; split partials are written in the same channel-blocked
// order (four consecutive channels of a lane are one 16-byte store).
// Single-buffer LDS of the channel-blocked kernel: the chunk buffer, or the
// output tile staged as [pixel][BN + 8 channels], whichever is larger.
template <class T>
__host__ __device__ constexpr size_t c8_one_buf_lds_bytes() {
  return (T::LDS_BUF > T::BM * (T::BN + 8) ? T::LDS_BUF : T::BM * (T::BN + 8)) * sizeof(u16);
}

// POOL (forward only): the unsplit output tile is not written; ReLU and 2x2
// max pooling run on it in LDS (bias added, rounded to bf16: the tensor the
// unfused forward would write), and the pooled tile and its window codes
// are written instead (a.out, a.pool_idx), as sb_relu_maxpool_fwd computes
// them from that tensor.
template <class T, bool DGRAD, bool ONE = false, bool POOL = false>
__global__ __launch_bounds__(256, 2) void conv3x3_c8_bf16(ConvArgs a) {
  static_assert(!(POOL && DGRAD), "pooling follows the forward pass");
  extern __shared__ u16 ldsb[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lc = lane & 31, lh = lane >> 5;

  int bt = blockIdx.x;
  const int tx = bt % a.tiles_w; bt /= a.tiles_w;
  const int ty = bt % a.tiles_h;
  const int tn = bt / a.tiles_h;
  const int n0 = tn * T::IMGS, h0 = ty * T::TH, w0 = tx * T::TW;
  const int co0 = blockIdx.y * T::BN;
  const int kc0 = blockIdx.z * a.chunks_per_split;
  const int kc1 = min(a.nchunks, kc0 + a.chunks_per_split);
  const int HWs = a.H * a.W;
  const int CB = a.Cin / 8;                          // input channel blocks

  // Halo staging: piece u = (channel block cb of the chunk, halo pixel hp),
  // halo pixels fastest.  Element offset of the piece for chunk 0 (from
  // image n0), -1 outside the image; a chunk adds 2 blocks of H*W pixels.
  constexpr int NP = 2 * T::PLANE;
  constexpr int XI = (NP + 255) / 256;
  int x_off[XI], x_cb[XI];
#pragma unroll
  for (int i = 0; i < XI; ++i) {
    const int u = tid + 256 * i;
    const int cb = u / T::PLANE, hp = u % T::PLANE;
    const int row = hp / T::HW, hx = hp % T::HW;
    const int img = row / T::HH, hy = row % T::HH;
    const int h = h0 + hy - 1, w = w0 + hx - 1;
    const bool ok = u < NP && n0 + img < a.N && (unsigned)h < (unsigned)a.H &&
                    (unsigned)w < (unsigned)a.W;
    x_off[i] = ok ? ((img * CB + cb) * HWs + h * a.W + w) * 8 : -1;
    x_cb[i] = u < NP ? cb : 1 << 20;
  }
  int b_off[T::MB];
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb) {
    const int p = wave * T::WP + mb * 32 + lc;
    b_off[mb] = (lh * T::PLANE + T::hp(T::img_of(p), T::yy_of(p), T::xx_of(p))) * 8;
  }

  f16 acc[T::NB][T::MB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i)
#pragma unroll
    for (int j = 0; j < T::MB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const rsrc_t xr = input_rsrc<u16>(a, n0, T::IMGS);
  const rsrc_t wr = packed_rsrc<u16, T::WTS>(a, blockIdx.y);
  s8 rx[XI];
  s8 rw[T::WTS_I];
  auto gload = [&](int kc) {
#pragma unroll
    for (int i = 0; i < XI; ++i) {
      const bool ok = x_off[i] >= 0 && 2 * kc + x_cb[i] < CB;
      const uint32_t off = ok ? (uint32_t)(x_off[i] + 2 * kc * HWs * 8) * 2u : kOOB;
      rx[i] = __builtin_bit_cast(s8, __builtin_amdgcn_raw_buffer_load_b128(xr, (int)off, 0, 0));
    }
#pragma unroll
    for (int i = 0; i < T::WTS_I; ++i) {
      const int g = tid + 256 * i;
      const uint32_t off = g < T::WTS_V ? (uint32_t)(kc * T::WTS + g * 8) * 2u : kOOB;
      rw[i] = __builtin_bit_cast(s8, __builtin_amdgcn_raw_buffer_load_b128(wr, (int)off, 0, 0));
    }
  };
  auto lstore = [&](int buf) {
    u16* X = ldsb + buf * T::LDS_BUF;
    u16* Wl = X + T::LDS_X;
#pragma unroll
    for (int i = 0; i < XI; ++i) {
      const int u = tid + 256 * i;
      if (u < NP) *reinterpret_cast<s8*>(X + u * 8) = rx[i];      // = [cb][halo pixel][8]
    }
#pragma unroll
    for (int i = 0; i < T::WTS_I; ++i) {
      const int g = tid + 256 * i;
      if (g < T::WTS_V) *reinterpret_cast<s8*>(Wl + g * 8) = rw[i];
    }
  };
  auto compute = [&](int buf) {
    const u16* X = ldsb + buf * T::LDS_BUF;
    const u16* Wl = X + T::LDS_X;
    // The operands of tap t + 1 are read before tap t's MFMAs are issued,
    // so each read has a whole tap's MFMAs to arrive under.
    s8 fa[2][T::NB], fb[2][T::MB];
    auto rd = [&](int t, int s) {
      const int toff = T::hp(0, t / 3, t % 3) * 8;
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
        fa[s][nb] = *reinterpret_cast<const s8*>(Wl + ((t * 2 + lh) * T::BN + nb * 32 + lc) * 8);
#pragma unroll
      for (int mb = 0; mb < T::MB; ++mb)
        fb[s][mb] = *reinterpret_cast<const s8*>(X + b_off[mb] + toff);
    };
    rd(0, 0);
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      if (t + 1 < 9) rd(t + 1, (t + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);   // keep those reads ahead of the MFMAs
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb)
          acc[nb][mb] = mfma32x32x16bf16(fa[t & 1][nb], fb[t & 1][mb], acc[nb][mb]);
    }
  };

  const int nk = kc1 - kc0;
  if constexpr (ONE) {
    if (nk > 0) {
      gload(kc0);
      lstore(0);
    }
    __syncthreads();
    for (int t = 0; t < nk; ++t) {
      if (t + 1 < nk) gload(kc0 + t + 1);
      compute(0);
      __syncthreads();
      if (t + 1 < nk) {
        lstore(0);
        __syncthreads();
      }
    }
  } else {
    if (nk > 0) {
      gload(kc0);
      lstore(0);
      if (nk > 1) gload(kc0 + 1);
    }
    __syncthreads();
    for (int t = 0; t < nk; ++t) {
      const int buf = t & 1;
      if (t + 1 < nk) lstore(buf ^ 1);
      if (t + 2 < nk) gload(kc0 + t + 2);
      compute(buf);
      __syncthreads();
    }
  }

  // acc[nb][mb] element v: output channel co0 + nb*32 + 8*(v/4) + 4*lh +
  // v%4 of pixel wave*WP + mb*32 + lc; the four elements v = 4q .. 4q+3 are
  // four consecutive channels of one 8-channel block.
  const int KB = a.Cout / 8;
  if (a.splits > 1) {
    float* mine = a.part + (size_t)blockIdx.z * a.N * a.Cout * HWs;
#pragma unroll
    for (int mb = 0; mb < T::MB; ++mb) {
      const int p = wave * T::WP + mb * 32 + lc;
      const int img = T::img_of(p), h = h0 + T::yy_of(p), w = w0 + T::xx_of(p);
      if (n0 + img >= a.N || h >= a.H || w >= a.W) continue;
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int co = co0 + nb * 32 + 8 * q;          // block start
          if (co >= a.Cout) continue;
          const size_t o = (((size_t)(n0 + img) * KB + co / 8) * HWs + h * a.W + w) * 8 + 4 * lh;
          *reinterpret_cast<f4*>(mine + o) =
              f4{acc[nb][mb][4 * q], acc[nb][mb][4 * q + 1], acc[nb][mb][4 * q + 2],
                 acc[nb][mb][4 * q + 3]};
        }
    }
    return;
  }
  // Unsplit: bias and ReLU, rounded to bf16, staged as [pixel][channel]
  // (row pitch BN + 8) and written as 16-byte pieces; piece q = (channel
  // block q / BM, pixel q % BM), so consecutive threads write consecutive
  // pixels of one block.
  constexpr int EP = T::BN + 8;
  static_assert(T::BM * EP * sizeof(u16) <= (ONE ? c8_one_buf_lds_bytes<T>() : T::LDS_BYTES),
                "output tile fits the staging LDS");
  u16* E = ldsb;
#pragma unroll
  for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int cl = nb * 32 + 8 * q + 4 * lh;           // channel within the tile
      float bv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        bv[e] = a.bias && co0 + cl + e < a.Cout ? a.bias[co0 + cl + e] : 0.f;
#pragma unroll
      for (int mb = 0; mb < T::MB; ++mb) {
        float r[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          r[e] = acc[nb][mb][4 * q + e] + bv[e];
          if (a.relu && !(r[e] > 0.f)) r[e] = 0.f;
        }
        typedef uint32_t u2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<u2*>(E + (wave * T::WP + mb * 32 + lc) * EP + cl) =
            u2{f32x2_to_bf16x2(r[0], r[1]), f32x2_to_bf16x2(r[2], r[3])};
      }
    }
  __syncthreads();
  if constexpr (POOL) {
    // Piece q = (channel block q / PP, pooled pixel q % PP): the window's
    // four 8-channel pieces come from LDS; per channel the first maximum in
    // row-major window order wins (strict >), the output is the maximum if
    // it is positive, else +0, and bit 7 of the code flags the latter.
    static_assert(T::TH % 2 == 0 && T::TW % 2 == 0, "whole 2x2 windows per tile");
    constexpr int PTH = T::TH / 2, PTW = T::TW / 2, PP = T::IMGS * PTH * PTW;
    constexpr int NPP = PP * (T::BN / 8);
    static_assert(NPP % 256 == 0, "whole rounds of pooled pieces");
    const int Hh = a.H / 2, Wh = a.W / 2;
    u16* yout = (u16*)a.out;
#pragma unroll
    for (int i = 0; i < NPP / 256; ++i) {
      const int q = tid + 256 * i;
      const int kb = q / PP, pp = q % PP;
      const int img = pp / (PTH * PTW), r = pp % (PTH * PTW);
      const int py = r / PTW, px = r % PTW;
      const int n = n0 + img, oh = h0 / 2 + py, ow = w0 / 2 + px, co = co0 + kb * 8;
      if (n >= a.N || oh >= Hh || ow >= Wh || co >= a.Cout) continue;
      const int p00 = (img * T::TH + 2 * py) * T::TW + 2 * px;
      const s8 v[4] = {*reinterpret_cast<const s8*>(E + p00 * EP + kb * 8),
                       *reinterpret_cast<const s8*>(E + (p00 + 1) * EP + kb * 8),
                       *reinterpret_cast<const s8*>(E + (p00 + T::TW) * EP + kb * 8),
                       *reinterpret_cast<const s8*>(E + (p00 + T::TW + 1) * EP + kb * 8)};
      s8 o;
      uint32_t codes[2] = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        short best = v[0][e];
        float m = bf16_to_f32((u16)best);
        uint32_t c = 0;
#pragma unroll
        for (int j = 1; j < 4; ++j) {
          const float f = bf16_to_f32((u16)v[j][e]);
          if (f > m) { m = f; best = v[j][e]; c = (uint32_t)j; }
        }
        const bool pos = m > 0.f;
        o[e] = pos ? best : (short)0;
        codes[e / 4] |= (c | (pos ? 0u : 0x80u)) << (8 * (e % 4));
      }
      const size_t off = ((((size_t)n * KB + co / 8) * Hh + oh) * Wh + ow) * 8;
      *reinterpret_cast<s8*>(yout + off) = o;
      *reinterpret_cast<uint2*>(a.pool_idx + off) = make_uint2(codes[0], codes[1]);
    }
    return;
  }
  constexpr int NPC = T::BM * (T::BN / 8);               // pieces per block
  constexpr int EPI = NPC / 256;
  static_assert(NPC % 256 == 0, "whole rounds of pieces");
  int goff[EPI];                                          // element offset, -1 outside
#pragma unroll
  for (int i = 0; i < EPI; ++i) {
    const int q = tid + 256 * i;
    const int p = q % T::BM, kb = q / T::BM;
    const int img = T::img_of(p), h = h0 + T::yy_of(p), w = w0 + T::xx_of(p);
    const int co = co0 + kb * 8;
    goff[i] = co < a.Cout && n0 + img < a.N && h < a.H && w < a.W
                  ? (((n0 + img) * KB + co / 8) * HWs + h * a.W + w) * 8 : -1;
  }
  s8 mk[EPI];
  if (a.mask) {
    const rsrc_t mr = make_rsrc(a.mask, (uint32_t)((size_t)a.N * a.Cout * HWs * 2));
#pragma unroll
    for (int i = 0; i < EPI; ++i) {
      const uint32_t off = goff[i] >= 0 ? (uint32_t)goff[i] * 2u : kOOB;
      mk[i] = __builtin_bit_cast(s8, __builtin_amdgcn_raw_buffer_load_b128(mr, (int)off, 0, 0));
    }
  }
  u16* out = (u16*)a.out;
#pragma unroll
  for (int i = 0; i < EPI; ++i) {
    if (goff[i] < 0) continue;
    const int q = tid + 256 * i;
    s8 o = *reinterpret_cast<const s8*>(E + (q % T::BM) * EP + (q / T::BM) * 8);
    if (a.mask) {
      // A bf16 mask value m keeps the output iff m > 0: bits 0x0001..0x7f80.
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t m16 = (uint16_t)mk[i][e];
        if (!(((m16 - 1u) & 0xffffu) < 0x7f80u)) o[e] = 0;
      }
    }
    *reinterpret_cast<s8*>(out + goff[i]) = o;
  }
}

// ---------------------------------------------------------------- host --
using BTileW32 = BTile<8, 32, 1>;
using BTileW16 = BTile<16, 16, 1>;
using BTileW8 = BTile<8, 8, 4>;
using BTileW32L = BTile<16, 32, 1>;     // 512 pixels: 64 x 128 per wave
using BTileW64L = BTile<8, 64, 1>;
using BTileW32N = BTile<8, 32, 1, 1>;   // 32 output channels (few-channel outputs)

static const char* kBTileNames[] = {
    "sb::conv3x3_igemm_bf16<sb::BTile<8, 32, 1>, %s, %d>",
    "sb::conv3x3_igemm_bf16<sb::BTile<16, 16, 1>, %s, %d>",
    "sb::conv3x3_igemm_bf16<sb::BTile<8, 8, 4>, %s, %d>",
    "sb::conv3x3_igemm_bf16<sb::BTile<16, 32, 1>, %s, %d>",
    "sb::conv3x3_igemm_bf16<sb::BTile<8, 64, 1>, %s, %d>",
    "sb::conv3x3_igemm_bf16<sb::BTile<8, 32, 1, 1>, %s, %d>",
};

struct BPlan {
  bool ok;
  int tile, imgs, grid_x, co_tiles, tiles_w, tiles_h, nchunks, cps, splits;
  size_t pack_bytes, part_off, ws_bytes;
};

// The bf16 MFMA path takes images at least 8 wide; narrower ones stay on the
// fp32-MFMA kernels.  Channel counts below the 16-channel chunk or the
// 64-channel output tile are padded (the first layer's 3 input channels,
// its data gradient's 3 output channels).  v8: the tensors allow 8-column
// staging, which the 512-pixel tiles need (their registers leave no room for
// the narrower staging).  The 512-pixel tiles pay off on long channel loops
// (256 or more input channels); with fewer chunks per block the 256-pixel
// tile's shorter prologue and epilogue win.
static BPlan bf16_plan(int N, int Cin, int H, int W, int Cout, bool v8) {
  BPlan p{};
  if (W < 8) return p;
  int th, tw, imgs = 1;
  // 512-pixel tiles (each wave 64 channels x 128 pixels: a quarter fewer LDS
  // operand bytes per MFMA than 64 x 64), 16 x 32 or 8 x 64, whichever pads
  // the image less, when they still fill the chip without a split.
  // (Never for outputs of 32 channels or fewer: their 32-channel tile's
  // filter layout must not depend on the tensors' alignment.)
  bool big = W >= 32 && v8 && Cin >= 256 && Cout > 32;
  if (big) {
    const long a16 = (long)round_up(H, 16) * round_up(W, 32);
    const long a8 = (long)round_up(H, 8) * round_up(W, 64);
    if (a16 <= a8) { p.tile = 3; th = 16; tw = 32; }
    else { p.tile = 4; th = 8; tw = 64; }
    big = (long)cdiv(W, tw) * cdiv(H, th) * N * cdiv(Cout, 64) >= 512;
  }
  if (!big) {
    if (W >= 32 && Cout <= 32) { p.tile = 5; th = 8; tw = 32; }
    else if (W >= 32) { p.tile = 0; th = 8; tw = 32; }
    else if (W >= 16) { p.tile = 1; th = 16; tw = 16; }
    else { p.tile = 2; th = 8; tw = 8; imgs = 4; }
  }
  p.ok = true;
  p.imgs = imgs;
  p.tiles_w = cdiv(W, tw);
  p.tiles_h = cdiv(H, th);
  p.grid_x = p.tiles_w * p.tiles_h * cdiv(N, imgs);
  const int bn = p.tile == 5 ? 32 : 64;
  p.co_tiles = cdiv(Cout, bn);
  p.nchunks = cdiv(Cin, 16);
  const long blocks = (long)p.grid_x * p.co_tiles;
  // About two resident blocks on each of the 256 CUs; at most 8 splits, and
  // at least two chunks per split.
  const long target = 512;
  int splits = 1;
  if (blocks < target)
    splits = (int)std::min<long>(std::min<long>(8, std::max(1, p.nchunks / 2)),
                                 cdiv((int)target, (int)blocks));
  p.cps = cdiv(p.nchunks, splits);
  p.splits = cdiv(p.nchunks, p.cps);
  p.pack_bytes = (size_t)p.co_tiles * p.nchunks * 9 * 16 * bn * sizeof(u16);
  p.part_off = round_up(p.pack_bytes, 256);
  p.ws_bytes = p.part_off +
               (p.splits > 1 ? (size_t)p.splits * N * Cout * H * W * sizeof(float) : 0);
  return p;
}

// Columns per halo load and per output / mask access: the largest of 8, 4,
// 2 that divides the image width and keeps every such access aligned, else 1.
static int bf16_vec(int W, const void* in, const void* out, const void* mask) {
  const uintptr_t u = (uintptr_t)in | (uintptr_t)out | (uintptr_t)mask;
  for (int v = 8; v >= 2; v /= 2)
    if (W % v == 0 && (u % (2 * v)) == 0) return v;
  return 1;
}

// Packs the filters of a layer for the bf16 kernels: [tap][ci/8][co][ci%8]
// slices of 16 input x BN output channels (BN = 32 for the 32-channel tile).
template <bool DGRAD>
static void bf16_pack(const BPlan& p, const void* wt, void* packed, int Cin, int Cout,
                      hipStream_t st) {
  if (p.tile == 5)
    filter_pack<DGRAD, 16, 32, u16, PackCI8><<<p.co_tiles * p.nchunks, 256, 0, st>>>(
        (const u16*)wt, (u16*)packed, Cin, Cout);
  else
    filter_pack<DGRAD, 16, 64, u16, PackCI8><<<p.co_tiles * p.nchunks, 256, 0, st>>>(
        (const u16*)wt, (u16*)packed, Cin, Cout);
}

// pack: the call packs the filters itself (into the workspace); otherwise
// a.wpk already holds them.
template <class T, bool DGRAD, int V>
static void bf16_launch(const BPlan& p, const ConvArgs& a, bool pack, hipStream_t st) {
  // Short channel loops (at most 8 chunks) on the 256-pixel tiles take the
  // single-buffer form.
  constexpr bool can_one = T::BM == 256;
  const bool one = can_one && p.cps <= 8;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)conv3x3_igemm_bf16<T, DGRAD, V>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
    if constexpr (can_one)
      (void)hipFuncSetAttribute((const void*)conv3x3_igemm_bf16<T, DGRAD, V, true>,
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)one_buf_lds_bytes<T>());
    attr_set = true;
  }
  if (pack) bf16_pack<DGRAD>(p, a.wt, (void*)a.wpk, a.Cin, a.Cout, st);
  dim3 grid(p.grid_x, p.co_tiles, p.splits);
  ConvArgs k = a;
  if (p.splits > 1) { k.bias = nullptr; k.mask = nullptr; k.relu = 0; }
  if constexpr (can_one) {
    if (one)
      conv3x3_igemm_bf16<T, DGRAD, V, true><<<grid, 256, one_buf_lds_bytes<T>(), st>>>(k);
    else
      conv3x3_igemm_bf16<T, DGRAD, V><<<grid, 256, T::LDS_BYTES, st>>>(k);
  } else {
    conv3x3_igemm_bf16<T, DGRAD, V><<<grid, 256, T::LDS_BYTES, st>>>(k);
  }
  if (p.splits > 1) {
    size_t total = (size_t)a.N * a.Cout * a.H * a.W;
    launch_splitk_reduce<u16>(a.part, p.splits, total, a.Cout, a.H * a.W, a.bias, a.relu,
                              (const u16*)a.mask, (u16*)a.out, st);
  }
}

template <class T, bool DGRAD>
static void bf16_launch_v(int v, const BPlan& p, const ConvArgs& a, bool pack, hipStream_t st) {
  switch (v) {
    case 8: bf16_launch<T, DGRAD, 8>(p, a, pack, st); break;
    case 4: bf16_launch<T, DGRAD, 4>(p, a, pack, st); break;
    case 2: bf16_launch<T, DGRAD, 2>(p, a, pack, st); break;
    default: bf16_launch<T, DGRAD, 1>(p, a, pack, st); break;
  }
}

template <bool DGRAD>
static void bf16_dispatch(int v, const BPlan& p, const ConvArgs& a, bool pack, hipStream_t st) {
  switch (p.tile) {
    case 0: bf16_launch_v<BTileW32, DGRAD>(v, p, a, pack, st); break;
    case 1: bf16_launch_v<BTileW16, DGRAD>(v, p, a, pack, st); break;
    case 2: bf16_launch_v<BTileW8, DGRAD>(v, p, a, pack, st); break;
    case 3: bf16_launch<BTileW32L, DGRAD, 8>(p, a, pack, st); break;
    case 4: bf16_launch<BTileW64L, DGRAD, 8>(p, a, pack, st); break;
    default: bf16_launch_v<BTileW32N, DGRAD>(v, p, a, pack, st); break;
  }
}

template <class T, bool DGRAD>
static void c8_launch(const BPlan& p, const ConvArgs& a, bool pack, hipStream_t st) {
  constexpr bool can_one = T::BM == 256;
  const bool one = can_one && p.cps <= 8;
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute((const void*)conv3x3_c8_bf16<T, DGRAD>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
    if constexpr (can_one)
      (void)hipFuncSetAttribute((const void*)conv3x3_c8_bf16<T, DGRAD, true>,
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)c8_one_buf_lds_bytes<T>());
    if constexpr (!DGRAD) {
      (void)hipFuncSetAttribute((const void*)conv3x3_c8_bf16<T, false, false, true>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
      if constexpr (can_one)
        (void)hipFuncSetAttribute((const void*)conv3x3_c8_bf16<T, false, true, true>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)c8_one_buf_lds_bytes<T>());
    }
  });
  if (pack) bf16_pack<DGRAD>(p, a.wt, (void*)a.wpk, a.Cin, a.Cout, st);
  dim3 grid(p.grid_x, p.co_tiles, p.splits);
  ConvArgs k = a;
  if (p.splits > 1) { k.bias = nullptr; k.mask = nullptr; k.relu = 0; }
  if constexpr (!DGRAD) {
    if (a.pool_idx) {                      // the caller checked: one split
      if (can_one && one)
        conv3x3_c8_bf16<T, false, true, true><<<grid, 256, c8_one_buf_lds_bytes<T>(), st>>>(k);
      else
        conv3x3_c8_bf16<T, false, false, true><<<grid, 256, T::LDS_BYTES, st>>>(k);
      return;
    }
  }
  if (can_one && one)
    conv3x3_c8_bf16<T, DGRAD, true><<<grid, 256, c8_one_buf_lds_bytes<T>(), st>>>(k);
  else
    conv3x3_c8_bf16<T, DGRAD><<<grid, 256, T::LDS_BYTES, st>>>(k);
  if (p.splits > 1) {
    size_t total = (size_t)a.N * a.Cout * a.H * a.W;
    launch_splitk_reduce<u16, true>(a.part, p.splits, total, a.Cout, a.H * a.W, a.bias,
                                    a.relu, (const u16*)a.mask, (u16*)a.out, st);
  }
}

template <bool DGRAD>
static void c8_dispatch(const BPlan& p, const ConvArgs& a, bool pack, hipStream_t st) {
  switch (p.tile) {
    case 0: c8_launch<BTileW32, DGRAD>(p, a, pack, st); break;
    case 1: c8_launch<BTileW16, DGRAD>(p, a, pack, st); break;
    case 2: c8_launch<BTileW8, DGRAD>(p, a, pack, st); break;
    case 3: c8_launch<BTileW32L, DGRAD>(p, a, pack, st); break;
    case 4: c8_launch<BTileW64L, DGRAD>(p, a, pack, st); break;
    default: c8_launch<BTileW32N, DGRAD>(p, a, pack, st); break;
  }
}

}  // namespace sb

namespace sbh {

// Workspace of the bf16 MFMA path (either staging width), or 0 when it does
// not take the shape.  prepacked: the filters come packed, the workspace
// holds only the split partials.
size_t conv_bf16_ws(int N, int Cin, int H, int W, int Cout, bool prepacked) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout, true);
  sb::BPlan q = sb::bf16_plan(N, Cin, H, W, Cout, false);
  if (!p.ok) return 0;
  if (prepacked) return std::max(p.ws_bytes - p.part_off, q.ws_bytes - q.part_off);
  return std::max(p.ws_bytes, q.ws_bytes);
}

// Bytes of the packed filters (the same for either staging width).
size_t conv_bf16_pack_bytes(int N, int Cin, int H, int W, int Cout) {
  return sb::bf16_plan(N, Cin, H, W, Cout, false).pack_bytes;
}

// Slice geometry of the packed filters: CK input x BN output channels per
// slice (PackCI8), `slices` slices.
void conv_bf16_pack_geom(int N, int Cin, int H, int W, int Cout, int* ck, int* bn, int* slices) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout, false);
  *ck = 16;
  *bn = p.tile == 5 ? 32 : 64;
  *slices = p.co_tiles * p.nchunks;
}

void conv_bf16_pack(bool dgrad, int N, int Cin, int H, int W, int Cout, const void* wt,
                    void* packed, hipStream_t st) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout, false);
  if (dgrad) sb::bf16_pack<true>(p, wt, packed, Cin, Cout, st);
  else sb::bf16_pack<false>(p, wt, packed, Cin, Cout, st);
}

bool conv_bf16_takes(int N, int Cin, int H, int W, int Cout) {
  return sb::bf16_plan(N, Cin, H, W, Cout, false).ok;
}

// Names the kernel as launched for aligned tensors.
int conv_bf16_describe(bool dgrad, int N, int Cin, int H, int W, int Cout, char* buf, size_t len) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout, W % 8 == 0);
  char name[160];
  snprintf(name, sizeof(name), sb::kBTileNames[p.tile], dgrad ? "true" : "false",
           sb::bf16_vec(W, nullptr, nullptr, nullptr));
  return snprintf(buf, len, "%s grid=%dx%dx%d", name, p.grid_x, p.co_tiles, p.splits);
}

sb_status conv_bf16(bool dgrad, int N, int Cin, int H, int W, int Cout, const void* in,
                    const void* wt, const float* bias, const void* mask, void* out, void* ws,
                    size_t ws_bytes, int relu, bool prepacked, hipStream_t st) {
  const int v = sb::bf16_vec(W, in, out, mask);
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout, v == 8);
  if (!p.ok) return SB_ERR_UNSUPPORTED;
  // Buffer ranges: one block's images of the input and of the output / mask,
  // one tile's packed filters.
  if ((int64_t)std::min(p.imgs, N) * std::max(Cin, Cout) * H * W * 2 >= (1ll << 31) ||
      (int64_t)p.pack_bytes >= (1ll << 31))
    return SB_ERR_UNSUPPORTED;
  const size_t part_off = prepacked ? 0 : p.part_off;
  const size_t need = prepacked ? p.ws_bytes - p.part_off : p.ws_bytes;
  if (need && (ws == nullptr || ws_bytes < need)) return SB_ERR_WORKSPACE;
  sb::ConvArgs a{};
  a.in = in; a.wt = wt; a.bias = bias; a.mask = mask; a.out = out;
  a.wpk = prepacked ? wt : ws;
  a.part = p.splits > 1 ? (float*)((char*)ws + part_off) : nullptr;
  a.N = N; a.Cin = Cin; a.H = H; a.W = W; a.Cout = Cout;
  a.tiles_w = p.tiles_w; a.tiles_h = p.tiles_h;
  a.nchunks = p.nchunks; a.chunks_per_split = p.cps; a.splits = p.splits; a.relu = relu;
  if (dgrad) sb::bf16_dispatch<true>(v, p, a, !prepacked, st);
  else sb::bf16_dispatch<false>(v, p, a, !prepacked, st);
  return launch_status();
}

// Channel-blocked bf16 tensors (SB_NCHW8C): the same plans (and filter
// packing) as the NCHW bf16 path with 16-byte staging.
int conv_bf16c8_describe(bool dgrad, int N, int Cin, int H, int W, int Cout, char* buf,
                         size_t len, bool pool) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout, true);
  static const char* kNames[] = {"8, 32, 1", "16, 16, 1", "8, 8, 4", "16, 32, 1", "8, 64, 1",
                                 "8, 32, 1, 1"};
  return snprintf(buf, len, "sb::conv3x3_c8_bf16<sb::BTile<%s>, %s%s> grid=%dx%dx%d",
                  kNames[p.tile], dgrad ? "true" : "false", pool ? ", pool" : "", p.grid_x,
                  p.co_tiles, p.splits);
}

// Whether the forward can pool its output in the kernel (fused ReLU + 2x2
// max pooling): even image sizes and an unsplit channel loop.
bool conv_bf16c8_pools(int N, int Cin, int H, int W, int Cout) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout, true);
  return p.ok && p.splits == 1 && H % 2 == 0 && W % 2 == 0;
}

// pool_idx: forward only; when given, `out` receives the pooled tensor
// [N][Cout/8][H/2][W/2][8] and pool_idx its codes (relu must be 0).
sb_status conv_bf16c8(bool dgrad, int N, int Cin, int H, int W, int Cout, const void* in,
                      const void* wt, const float* bias, const void* mask, void* out, void* ws,
                      size_t ws_bytes, int relu, bool prepacked, hipStream_t st,
                      uint8_t* pool_idx) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout, true);
  if (!p.ok) return SB_ERR_UNSUPPORTED;
  if (pool_idx && (dgrad || relu || !conv_bf16c8_pools(N, Cin, H, W, Cout)))
    return SB_ERR_UNSUPPORTED;
  // Buffer ranges: the whole output (mask) tensor, one block's images of the
  // input, one tile's packed filters.
  if ((int64_t)N * std::max(Cin, Cout) * H * W * 2 >= (1ll << 31) ||
      (int64_t)p.pack_bytes >= (1ll << 31))
    return SB_ERR_UNSUPPORTED;
  const size_t part_off = prepacked ? 0 : p.part_off;
  const size_t need = prepacked ? p.ws_bytes - p.part_off : p.ws_bytes;
  if (need && (ws == nullptr || ws_bytes < need)) return SB_ERR_WORKSPACE;
  sb::ConvArgs a{};
  a.in = in; a.wt = wt; a.bias = bias; a.mask = mask; a.out = out;
  a.wpk = prepacked ? wt : ws;
  a.part = p.splits > 1 ? (float*)((char*)ws + part_off) : nullptr;
  a.N = N; a.Cin = Cin; a.H = H; a.W = W; a.Cout = Cout;
  a.tiles_w = p.tiles_w; a.tiles_h = p.tiles_h;
  a.nchunks = p.nchunks; a.chunks_per_split = p.cps; a.splits = p.splits; a.relu = relu;
  a.pool_idx = pool_idx;
  if (dgrad) sb::c8_dispatch<true>(p, a, !prepacked, st);
  else sb::c8_dispatch<false>(p, a, !prepacked, st);
  return launch_status();
}

}  // namespace sbh
