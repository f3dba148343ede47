// conv_bf16.hip -- 3x3 / stride 1 / pad 1 convolution forward and data
// gradient with bf16 operands on the bf16 MFMA (v_mfma_f32_16x16x16_bf16,
// fp32 accumulation), for SB_BF16 tensors.
//
// The same implicit GEMM as the fp32 kernels (rows = output channels,
// columns = 128 output pixels, reduction = input channels x 9 taps, the
// input halo of a chunk staged once in LDS and read at 9 shifted windows),
// with both operands held channel-innermost in LDS, because a lane of this
// MFMA supplies 4 consecutive reduction values (4 consecutive input
// channels at one tap):
//   * filters, packed per (output-channel tile, 16-channel chunk) as
//     [tap][co][ci] (filter_pack with CI_INNER); LDS rows of 16 ci;
//   * input halo, transposed on its way into LDS from NCHW to
//     [halo pixel][ci].
// LDS rows are 24 bf16 (48 bytes = 12 banks) apart, so the 16 lanes of a
// lane group, reading 8 bytes from 16 consecutive rows, touch 16 distinct
// 4-bank groups: the operand reads are conflict-free.  Each MFMA consumes
// one 8-byte read per operand.
//
// The data gradient is the same contraction with the filters transposed and
// rotated (done by the pack).  Splits over channel chunks, the epilogue and
// the split reduction are the fp32 path's.
#include "conv_common.hpp"

#include <algorithm>
#include <cstdio>

namespace sb {

typedef short s4 __attribute__((ext_vector_type(4)));

// D(16x16) += A(16x16) * B(16x16), bf16 in / fp32 accumulate.  Lane l
// supplies A[l%16][4*(l/16) + j] and B[4*(l/16) + j][l%16] (j = 0..3) and
// receives D[4*(l/16) + i][l%16] in element i.
__device__ __forceinline__ f4 mfma16x16x16bf16(s4 a, s4 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

template <int TH_, int TW_, int IMGS_>
struct BTile {
  static constexpr int TH = TH_, TW = TW_, IMGS = IMGS_;
  static constexpr int BM = IMGS * TH * TW;
  static_assert(BM == 128, "pixel tile must hold 128 pixels");
  static constexpr int BN = 64, CK = 16, RP = 24;   // RP: LDS row pitch (bf16)
  static constexpr int HH = TH + 2, HW = TW + 2;
  static constexpr int PLANE = IMGS * HH * HW;      // halo pixels
  static constexpr int HALO = CK * PLANE;           // halo elements per chunk
  static constexpr int HALO_PT = (HALO + 255) / 256;
  static constexpr int WTS = 9 * BN * CK;           // filter elements per chunk
  static constexpr int WTS_PT = WTS / 4 / 256;      // 8-byte groups per thread
  static_assert(WTS % 1024 == 0, "whole 256-thread rounds of 4-element groups");
  static constexpr int LDS_X = PLANE * RP;          // bf16 elements
  static constexpr int LDS_W = 9 * BN * RP;
  static constexpr int LDS_SPARE = 256;             // idle halo lanes store here
  static constexpr int LDS_BUF = LDS_X + LDS_W + LDS_SPARE;
  static_assert(LDS_X % 8 == 0 && LDS_BUF % 8 == 0, "8-byte aligned regions");
  static constexpr size_t LDS_BYTES = 2 * LDS_BUF * sizeof(u16);
  static_assert(LDS_BYTES <= 80 * 1024, "two blocks must fit in the 160 KB of LDS");
  // Four waves 2 x 2; a wave owns 32 channels x 64 pixels (2 x 4 blocks).
  static constexpr int WN = 32, WM = 64, NB = 2, MB = 4;
  // Halo layout [halo row][halo column][image] (image innermost), as the
  // fp32 tiles: the 16 pixels of an MFMA column block are consecutive rows.
  __host__ __device__ static constexpr int hoff(int img, int hy, int hx) {
    return (hy * HW + hx) * IMGS + img;
  }
  __device__ static void pix(int p, int& img, int& yy, int& xx) {
    img = p % IMGS;
    const int q = p / IMGS;
    yy = q / TW;
    xx = q - yy * TW;
  }
};

template <class T, bool DGRAD>
__global__ __launch_bounds__(256, 2) void conv3x3_igemm_bf16(ConvArgs a) {
  extern __shared__ u16 ldsb[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int kq = lane >> 4, lr = lane & 15;

  int bt = blockIdx.x;
  const int tx = bt % a.tiles_w; bt /= a.tiles_w;
  const int ty = bt % a.tiles_h;
  const int tn = bt / a.tiles_h;
  const int n0 = tn * T::IMGS, h0 = ty * T::TH, w0 = tx * T::TW;
  const int co0 = blockIdx.y * T::BN;
  const int kc0 = blockIdx.z * a.chunks_per_split;
  const int kc1 = min(a.nchunks, kc0 + a.chunks_per_split);
  const int HWs = a.H * a.W;

  // Halo element e = (channel cc, halo position rem), position fastest, so
  // that neighbouring lanes read neighbouring pixels of one channel plane.
  int x_off[T::HALO_PT], x_c[T::HALO_PT], x_loff[T::HALO_PT];
#pragma unroll
  for (int i = 0; i < T::HALO_PT; ++i) {
    int e = tid + i * 256;
    bool live = e < T::HALO;
    int cc = e / T::PLANE, rem = e - cc * T::PLANE;
    int img = rem % T::IMGS, q = rem / T::IMGS;
    int yy = q / T::HW, xx = q - yy * T::HW;
    int n = n0 + img, h = h0 + yy - 1, w = w0 + xx - 1;
    bool ok = live && n < a.N && h >= 0 && h < a.H && w >= 0 && w < a.W;
    x_off[i] = ok ? img * a.Cin * HWs + h * a.W + w : -1;   // from image n0; + ci * H*W
    x_c[i] = cc;
    x_loff[i] = live ? rem * T::RP + cc : T::LDS_X + T::LDS_W + tid;
  }
  // Packed filter group g (4 consecutive ci of one (tap, co) row) -> LDS.
  int w_loff[T::WTS_PT];
#pragma unroll
  for (int i = 0; i < T::WTS_PT; ++i) {
    int g = tid + i * 256;
    w_loff[i] = (g >> 2) * T::RP + (g & 3) * 4;
  }
  int pix_off[T::MB];
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb) {
    int img, yy, xx;
    T::pix(wm * T::WM + mb * 16 + lr, img, yy, xx);
    pix_off[mb] = T::hoff(img, yy, xx) * T::RP + 4 * kq;
  }

  f4 acc[T::NB][T::MB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i)
#pragma unroll
    for (int j = 0; j < T::MB; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  const rsrc_t xr = input_rsrc<u16>(a, n0, T::IMGS);
  const rsrc_t wr = packed_rsrc<u16, T::WTS>(a, blockIdx.y);
  u16 rx[T::HALO_PT];
  s4 rw[T::WTS_PT];
  auto gload = [&](int kc) {
    const int cbase = kc * T::CK;
#pragma unroll
    for (int i = 0; i < T::HALO_PT; ++i) {
      const int ci = cbase + x_c[i];
      const bool ok = x_off[i] >= 0 && ci < a.Cin;
      rx[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(
          xr, ok ? (int)((uint32_t)(x_off[i] + ci * HWs) * 2u) : (int)kOOB, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < T::WTS_PT; ++i)
      rw[i] = __builtin_bit_cast(
          s4, __builtin_amdgcn_raw_buffer_load_b64(
                  wr, (int)((uint32_t)(kc * T::WTS + (tid + i * 256) * 4) * 2u), 0, 0));
  };
  auto lstore = [&](int buf) {
    u16* X = ldsb + buf * T::LDS_BUF;
    u16* Wl = X + T::LDS_X;
#pragma unroll
    for (int i = 0; i < T::HALO_PT; ++i) X[x_loff[i]] = rx[i];
#pragma unroll
    for (int i = 0; i < T::WTS_PT; ++i) *reinterpret_cast<s4*>(Wl + w_loff[i]) = rw[i];
  };
  auto compute = [&](int buf) {
    const u16* X = ldsb + buf * T::LDS_BUF;
    const u16* Wl = X + T::LDS_X;
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int toff = T::hoff(0, t / 3, t % 3) * T::RP;
      s4 fa[T::NB], fb[T::MB];
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
        fa[nb] = *reinterpret_cast<const s4*>(
            Wl + (t * T::BN + wn * T::WN + nb * 16 + lr) * T::RP + 4 * kq);
#pragma unroll
      for (int mb = 0; mb < T::MB; ++mb)
        fb[mb] = *reinterpret_cast<const s4*>(X + pix_off[mb] + toff);
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb)
          acc[nb][mb] = mfma16x16x16bf16(fa[nb], fb[mb], acc[nb][mb]);
    }
  };

  const int nk = kc1 - kc0;
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

  // acc[nb][mb] lane holds channel co0 + wn*WN + nb*16 + 4*kq + i of pixel
  // wm*WM + mb*16 + lr.
  const size_t total = (size_t)a.N * a.Cout * HWs;
  if (a.splits > 1) {
    float* mine = a.part + (size_t)blockIdx.z * total;
#pragma unroll
    for (int mb = 0; mb < T::MB; ++mb) {
      int img, yy, xx;
      T::pix(wm * T::WM + mb * 16 + lr, img, yy, xx);
      const int n = n0 + img, h = h0 + yy, w = w0 + xx;
      if (n >= a.N || h >= a.H || w >= a.W) continue;
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int co = co0 + wn * T::WN + nb * 16 + kq * 4 + i;
          if (co < a.Cout) mine[((size_t)n * a.Cout + co) * HWs + (size_t)h * a.W + w] =
              acc[nb][mb][i];
        }
    }
    return;
  }
  // Element offsets from image n0 (the output and the ReLU mask share the
  // layout); -1 outside the tensor.  The mask values are all requested
  // before any is used.
  int off[T::MB][T::NB][4];
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb) {
    int img, yy, xx;
    T::pix(wm * T::WM + mb * 16 + lr, img, yy, xx);
    const bool pix_ok = n0 + img < a.N && h0 + yy < a.H && w0 + xx < a.W;
#pragma unroll
    for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int co = co0 + wn * T::WN + nb * 16 + kq * 4 + i;
        off[mb][nb][i] = pix_ok && co < a.Cout
                             ? (img * a.Cout + co) * HWs + (h0 + yy) * a.W + w0 + xx : -1;
      }
  }
  float mv[T::MB][T::NB][4];
  if (a.mask) {
    const int cnt = min(T::IMGS, a.N - n0);
    const rsrc_t mr = make_rsrc((const u16*)a.mask + (size_t)n0 * a.Cout * HWs,
                                (uint32_t)((size_t)cnt * a.Cout * HWs * 2));
#pragma unroll
    for (int mb = 0; mb < T::MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          mv[mb][nb][i] = BufLoad<u16>::one(
              mr, off[mb][nb][i] >= 0 ? (uint32_t)off[mb][nb][i] * 2u : kOOB);
  }
  u16* out = (u16*)a.out + (size_t)n0 * a.Cout * HWs;
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (off[mb][nb][i] < 0) continue;
        const int co = co0 + wn * T::WN + nb * 16 + kq * 4 + i;
        float v = acc[nb][mb][i];
        if (a.bias) v += a.bias[co];
        if (a.relu && !(v > 0.f)) v = 0.f;
        if (a.mask && !(mv[mb][nb][i] > 0.f)) v = 0.f;
        out[off[mb][nb][i]] = f32_to_bf16(v);
      }
}

// ---------------------------------------------------------------- host --
using BTileW32 = BTile<4, 32, 1>;
using BTileW16 = BTile<8, 16, 1>;
using BTileW8 = BTile<8, 8, 2>;

static const char* kBTileNames[] = {
    "sb::conv3x3_igemm_bf16<sb::BTile<4, 32, 1>, %s>",
    "sb::conv3x3_igemm_bf16<sb::BTile<8, 16, 1>, %s>",
    "sb::conv3x3_igemm_bf16<sb::BTile<8, 8, 2>, %s>",
};

struct BPlan {
  bool ok;
  int tile, imgs, grid_x, co_tiles, tiles_w, tiles_h, nchunks, cps, splits;
  size_t pack_bytes, part_off, ws_bytes;
};

// The bf16 MFMA path takes images at least 8 wide with at least 16 input
// channels; other shapes stay on the fp32-MFMA kernels.
static BPlan bf16_plan(int N, int Cin, int H, int W, int Cout) {
  BPlan p{};
  if (W < 8 || Cin < 16) return p;
  int th, tw, imgs = 1;
  if (W >= 32) { p.tile = 0; th = 4; tw = 32; }
  else if (W >= 16) { p.tile = 1; th = 8; tw = 16; }
  else { p.tile = 2; th = 8; tw = 8; imgs = 2; }
  p.ok = true;
  p.imgs = imgs;
  p.tiles_w = cdiv(W, tw);
  p.tiles_h = cdiv(H, th);
  p.grid_x = p.tiles_w * p.tiles_h * cdiv(N, imgs);
  p.co_tiles = cdiv(Cout, 64);
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
  p.pack_bytes = (size_t)p.co_tiles * p.nchunks * 9 * 16 * 64 * sizeof(u16);
  p.part_off = round_up(p.pack_bytes, 256);
  p.ws_bytes = p.part_off +
               (p.splits > 1 ? (size_t)p.splits * N * Cout * H * W * sizeof(float) : 0);
  return p;
}

template <class T, bool DGRAD>
static void bf16_launch(const BPlan& p, const ConvArgs& a, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)conv3x3_igemm_bf16<T, DGRAD>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
    attr_set = true;
  }
  filter_pack<DGRAD, T::CK, T::BN, u16, true><<<p.co_tiles * p.nchunks, 256, 0, st>>>(
      (const u16*)a.wt, (u16*)a.wpk, a.Cin, a.Cout);
  dim3 grid(p.grid_x, p.co_tiles, p.splits);
  ConvArgs k = a;
  if (p.splits > 1) { k.bias = nullptr; k.mask = nullptr; k.relu = 0; }
  conv3x3_igemm_bf16<T, DGRAD><<<grid, 256, T::LDS_BYTES, st>>>(k);
  if (p.splits > 1) {
    size_t total = (size_t)a.N * a.Cout * a.H * a.W;
    conv_splitk_reduce<u16><<<(unsigned)((total + 63) / 64), 256, 0, st>>>(
        a.part, p.splits, total, a.Cout, a.H * a.W, a.bias, a.relu, (const u16*)a.mask,
        (u16*)a.out);
  }
}

template <bool DGRAD>
static void bf16_dispatch(const BPlan& p, const ConvArgs& a, hipStream_t st) {
  switch (p.tile) {
    case 0: bf16_launch<BTileW32, DGRAD>(p, a, st); break;
    case 1: bf16_launch<BTileW16, DGRAD>(p, a, st); break;
    default: bf16_launch<BTileW8, DGRAD>(p, a, st); break;
  }
}

}  // namespace sb

namespace sbh {

// Workspace of the bf16 MFMA path, or 0 when it does not take the shape.
size_t conv_bf16_ws(int N, int Cin, int H, int W, int Cout) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout);
  return p.ok ? p.ws_bytes : 0;
}

bool conv_bf16_takes(int N, int Cin, int H, int W, int Cout) {
  return sb::bf16_plan(N, Cin, H, W, Cout).ok;
}

int conv_bf16_describe(bool dgrad, int N, int Cin, int H, int W, int Cout, char* buf, size_t len) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout);
  char name[160];
  snprintf(name, sizeof(name), sb::kBTileNames[p.tile], dgrad ? "true" : "false");
  return snprintf(buf, len, "%s grid=%dx%dx%d", name, p.grid_x, p.co_tiles, p.splits);
}

sb_status conv_bf16(bool dgrad, int N, int Cin, int H, int W, int Cout, const void* in,
                    const void* wt, const float* bias, const void* mask, void* out, void* ws,
                    size_t ws_bytes, int relu, hipStream_t st) {
  sb::BPlan p = sb::bf16_plan(N, Cin, H, W, Cout);
  if (!p.ok) return SB_ERR_UNSUPPORTED;
  // Buffer ranges: one block's images of the input and of the output / mask,
  // one tile's packed filters.
  if ((int64_t)std::min(p.imgs, N) * std::max(Cin, Cout) * H * W * 2 >= (1ll << 31) ||
      (int64_t)p.pack_bytes >= (1ll << 31))
    return SB_ERR_UNSUPPORTED;
  if (ws == nullptr || ws_bytes < p.ws_bytes) return SB_ERR_WORKSPACE;
  sb::ConvArgs a{};
  a.in = in; a.wt = wt; a.bias = bias; a.mask = mask; a.out = out;
  a.wpk = ws;
  a.part = p.splits > 1 ? (float*)((char*)ws + p.part_off) : nullptr;
  a.N = N; a.Cin = Cin; a.H = H; a.W = W; a.Cout = Cout;
  a.tiles_w = p.tiles_w; a.tiles_h = p.tiles_h;
  a.nchunks = p.nchunks; a.chunks_per_split = p.cps; a.splits = p.splits; a.relu = relu;
  if (dgrad) sb::bf16_dispatch<true>(p, a, st);
  else sb::bf16_dispatch<false>(p, a, st);
  return launch_status();
}

}  // namespace sbh
