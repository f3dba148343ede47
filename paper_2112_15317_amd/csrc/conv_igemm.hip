// conv_igemm.hip -- 3x3 / stride 1 / pad 1 convolution forward and data
// gradient as an implicit GEMM on fp32 MFMA (v_mfma_f32_16x16x4_f32).
//
// Forward (sec. 2.2): out[n,co,h,w] = sum_{ci,r,s} in[n,ci,h+r-1,w+s-1] * w[co,ci,r,s].
// The data gradient is the same contraction with the filters transposed
// (co <-> ci) and rotated by 180 degrees: dx[n,c,i,j] = sum_{k,r,s}
// dy[n,k,i+r-1,j+s-1] * w[k,c,2-r,2-s].  One kernel serves both; only the
// filter gather differs.
//
// GEMM view per block: rows = BN output channels, columns = BM = 128 output
// pixels (IMGS images x TH rows x TW cols), reduction = input channels x 9
// taps.  For each chunk of CK input channels the block stages in LDS
//   * the input halo: CK x IMGS x (TH+2) x (TW+2) values, read once from HBM
//     and reused by all 9 taps (a shifted window per tap, no im2col), and
//   * the filter slice: 9 x CK x BN values, laid out [tap][ci][co].
// The chunk loop is double-buffered: the global loads of chunk t+1 are in
// flight (in registers) while chunk t is multiplied out of LDS.
// Four waves split the tile 2 (channels) x 2 (pixels); each wave owns
// (BN/2) x 64 outputs = (BN/32) x 4 MFMA 16x16 blocks in AGPR/VGPR
// accumulators.  MFMA rows are channels and columns pixels so that the 16
// lanes of an output row store 16 consecutive pixels (coalesced NCHW).
//
// When the output grid alone cannot fill the 256 CUs (small late layers),
// the channel chunks are split over gridDim.z; each split writes raw sums to
// the workspace and conv_splitk_reduce adds them in a fixed order and applies
// the epilogue (bias + ReLU, or the ReLU mask of the layer below).
#include "sb_internal.hpp"

#include <algorithm>
#include <cstdio>

namespace sb {

template <int TH_, int TW_, int IMGS_, int CK_, int BN_>
struct ConvTile {
  static constexpr int TH = TH_, TW = TW_, IMGS = IMGS_, CK = CK_, BN = BN_;
  static constexpr int BM = IMGS * TH * TW;
  static_assert(BM == 128, "pixel tile must hold 128 pixels");
  static constexpr int HH = TH + 2, HW = TW + 2;
  static constexpr int PLANE = IMGS * HH * HW;
  // Channel stride of the halo in LDS: a multiple of 64 floats plus 16, so
  // the four k-rows an MFMA operand read touches land in different banks.
  static constexpr int PLANE_P = (PLANE + 63) / 64 * 64 + 16;
  // Row stride of the filter slice in LDS: 16 for BN = 16 (four k-rows fill
  // 64 consecutive banks), otherwise BN plus 16 (= 16 mod 64).
  static constexpr int BN_P = BN == 16 ? 16 : BN + 16;
  static constexpr int HALO = CK * PLANE;
  static constexpr int WTS = 9 * CK * BN;
  static constexpr int HALO_PT = (HALO + 255) / 256;
  static constexpr int WTS_PT = (WTS + 255) / 256;
  static constexpr int LDS_X = CK * PLANE_P;
  static constexpr int LDS_W = 9 * CK * BN_P;
  static constexpr int LDS_BUF = LDS_X + LDS_W;
  // Waves split the tile 2 x 2 (BN >= 32) or 1 x 4 along pixels (BN = 16).
  static constexpr int WAVES_N = BN >= 32 ? 2 : 1, WAVES_M = 4 / WAVES_N;
  static constexpr int WN = BN / WAVES_N, WM = BM / WAVES_M;
  static constexpr int NB = WN / 16, MB = WM / 16;
  static constexpr size_t LDS_BYTES = 2 * LDS_BUF * sizeof(float);
  static_assert(LDS_BYTES <= 80 * 1024, "two blocks must fit in the 160 KB of LDS");
};

template <class T, bool DGRAD>
__global__ __launch_bounds__(256, 2) void conv3x3_igemm_f32(
    const float* __restrict__ in, const float* __restrict__ wt,
    const float* __restrict__ bias, const float* __restrict__ mask,
    float* __restrict__ out, int N, int Cin, int H, int W, int Cout,
    int tiles_w, int tiles_h, int chunks_per_split, int relu, int partial) {
  extern __shared__ float lds[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % T::WAVES_M, wn = wave / T::WAVES_M;
  const int kq = lane >> 4, lr = lane & 15;

  int bt = blockIdx.x;
  const int tx = bt % tiles_w; bt /= tiles_w;
  const int ty = bt % tiles_h;
  const int tn = bt / tiles_h;
  const int n0 = tn * T::IMGS, h0 = ty * T::TH, w0 = tx * T::TW;
  const int co0 = blockIdx.y * T::BN;
  const int nchunks = cdiv(Cin, T::CK);
  const int kc0 = blockIdx.z * chunks_per_split;
  const int kc1 = min(nchunks, kc0 + chunks_per_split);
  const size_t HWs = (size_t)H * W;

  // ---- per-thread gather plan (independent of the chunk) ----
  // Halo element e of a chunk = (channel-in-chunk c, image, halo row, halo
  // col); its global address is x_base[i] + (chunk*CK + c) * H*W.
  size_t x_base[T::HALO_PT];
  int x_c[T::HALO_PT], x_loff[T::HALO_PT];
  bool x_ok[T::HALO_PT];
#pragma unroll
  for (int i = 0; i < T::HALO_PT; ++i) {
    int e = tid + i * 256;
    bool live = e < T::HALO;
    int c = e / T::PLANE, rem = e - c * T::PLANE;
    int img = rem / (T::HH * T::HW), r2 = rem - img * (T::HH * T::HW);
    int yy = r2 / T::HW, xx = r2 - yy * T::HW;
    int n = n0 + img, h = h0 + yy - 1, w = w0 + xx - 1;
    x_ok[i] = live && n < N && h >= 0 && h < H && w >= 0 && w < W;
    x_c[i] = c;
    x_base[i] = x_ok[i] ? (size_t)n * Cin * HWs + (size_t)h * W + w : 0;
    x_loff[i] = live ? c * T::PLANE_P + rem : -1;
  }

  int w_goff[T::WTS_PT], w_loff[T::WTS_PT], w_ci[T::WTS_PT];
  bool w_ok[T::WTS_PT];
#pragma unroll
  for (int i = 0; i < T::WTS_PT; ++i) {
    int e = tid + i * 256;
    bool live = e < T::WTS;
    if (!DGRAD) {
      // global order [co][ci][tap] -> LDS [tap][ci][co]
      int nn = e / (T::CK * 9), rem = e - nn * (T::CK * 9);
      int cc = rem / 9, tap = rem - cc * 9;
      int co = co0 + nn;
      w_ok[i] = live && co < Cout;
      w_ci[i] = cc;
      w_goff[i] = (co * Cin + cc) * 9 + tap;     // + chunk * CK * 9
      w_loff[i] = live ? (tap * T::CK + cc) * T::BN_P + nn : -1;
    } else {
      // forward filters [k][c][tap] with k = this conv's input channel:
      // global order [ci][co][tap] -> LDS [8 - tap][ci][co]
      int kk = e / (T::BN * 9), rem = e - kk * (T::BN * 9);
      int nn = rem / 9, tap = rem - nn * 9;
      int co = co0 + nn;
      w_ok[i] = live && co < Cout;
      w_ci[i] = kk;
      w_goff[i] = (kk * Cout + co) * 9 + tap;    // + chunk * CK * Cout * 9
      w_loff[i] = live ? ((8 - tap) * T::CK + kk) * T::BN_P + nn : -1;
    }
  }

  // ---- per-lane operand offsets ----
  int pix_off[T::MB];
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb) {
    int p = wm * T::WM + mb * 16 + lr;
    int img = p / (T::TH * T::TW), r = p - img * (T::TH * T::TW);
    int yy = r / T::TW, xx = r - yy * T::TW;
    pix_off[mb] = img * T::HH * T::HW + yy * T::HW + xx;
  }

  f4 acc[T::NB][T::MB];
#pragma unroll
  for (int a = 0; a < T::NB; ++a)
#pragma unroll
    for (int b = 0; b < T::MB; ++b) acc[a][b] = f4{0.f, 0.f, 0.f, 0.f};

  float rx[T::HALO_PT], rw[T::WTS_PT];

  auto gload = [&](int kc) {
    const int cbase = kc * T::CK;
#pragma unroll
    for (int i = 0; i < T::HALO_PT; ++i) {
      int ci = cbase + x_c[i];
      rx[i] = (x_ok[i] && ci < Cin) ? in[x_base[i] + (size_t)ci * HWs] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < T::WTS_PT; ++i) {
      int ci = cbase + w_ci[i];
      size_t off = DGRAD ? (size_t)w_goff[i] + (size_t)cbase * Cout * 9
                         : (size_t)w_goff[i] + (size_t)cbase * 9;
      rw[i] = (w_ok[i] && ci < Cin) ? wt[off] : 0.f;
    }
  };
  auto lstore = [&](int buf) {
    float* X = lds + buf * T::LDS_BUF;
    float* Wl = X + T::LDS_X;
#pragma unroll
    for (int i = 0; i < T::HALO_PT; ++i)
      if (x_loff[i] >= 0) X[x_loff[i]] = rx[i];
#pragma unroll
    for (int i = 0; i < T::WTS_PT; ++i)
      if (w_loff[i] >= 0) Wl[w_loff[i]] = rw[i];
  };

  if (kc0 < kc1) {
    gload(kc0);
    lstore(0);
  }
  __syncthreads();

  for (int kc = kc0; kc < kc1; ++kc) {
    const int buf = (kc - kc0) & 1;
    const bool more = kc + 1 < kc1;
    if (more) gload(kc + 1);
    const float* X = lds + buf * T::LDS_BUF;
    const float* Wl = X + T::LDS_X;
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      const int toff = (tap / 3) * T::HW + (tap % 3);
#pragma unroll
      for (int cg = 0; cg < T::CK / 4; ++cg) {
        float a[T::NB], b[T::MB];
#pragma unroll
        for (int nb = 0; nb < T::NB; ++nb)
          a[nb] = Wl[(tap * T::CK + cg * 4 + kq) * T::BN_P + wn * T::WN + nb * 16 + lr];
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb)
          b[mb] = X[(cg * 4 + kq) * T::PLANE_P + pix_off[mb] + toff];
#pragma unroll
        for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
          for (int mb = 0; mb < T::MB; ++mb)
            acc[nb][mb] = mfma16x16x4(a[nb], b[mb], acc[nb][mb]);
      }
    }
    if (more) lstore(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue ----
  const size_t split_off = partial ? (size_t)blockIdx.z * N * Cout * HWs : 0;
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb) {
    int p = wm * T::WM + mb * 16 + lr;
    int img = p / (T::TH * T::TW), r = p - img * (T::TH * T::TW);
    int yy = r / T::TW, xx = r - yy * T::TW;
    int n = n0 + img, h = h0 + yy, w = w0 + xx;
    if (n >= N || h >= H || w >= W) continue;
#pragma unroll
    for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int co = co0 + wn * T::WN + nb * 16 + kq * 4 + i;
        if (co >= Cout) continue;
        size_t off = ((size_t)n * Cout + co) * HWs + (size_t)h * W + w;
        float v = acc[nb][mb][i];
        if (partial) {
          out[split_off + off] = v;
        } else {
          if (bias) v += bias[co];
          if (relu && !(v > 0.f)) v = 0.f;
          if (mask && !(mask[off] > 0.f)) v = 0.f;
          out[off] = v;
        }
      }
  }
}

// Sum of the split partials in a fixed order, then the epilogue.
__global__ __launch_bounds__(256) void conv_splitk_reduce(
    const float* __restrict__ part, int splits, size_t total, int Cout, size_t HWs,
    const float* __restrict__ bias, int relu, const float* __restrict__ mask,
    float* __restrict__ out) {
  __shared__ float lds[256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t i = (size_t)blockIdx.x * 64 + lane;
  float v = SplitSum{part, splits, total}(i, wave, lds, lane);
  if (wave != 0 || i >= total) return;
  if (bias) v += bias[(i / HWs) % Cout];
  if (relu && !(v > 0.f)) v = 0.f;
  if (mask && !(mask[i] > 0.f)) v = 0.f;
  out[i] = v;
}

// ---------------------------------------------------------------- host --
struct IgemmPlan {
  int tile;          // index into the tile table
  int tiles_w, tiles_h, tiles_n, co_tiles;
  int nchunks, cps, splits;
  size_t ws_bytes;
};

using TileW32 = ConvTile<4, 32, 1, 8, 64>;
using TileW16 = ConvTile<8, 16, 1, 8, 64>;
using TileW8 = ConvTile<8, 8, 2, 8, 64>;
using TileW4 = ConvTile<4, 4, 8, 8, 64>;
using TileW2 = ConvTile<2, 2, 32, 8, 64>;
using TileW32c4 = ConvTile<4, 32, 1, 4, 64>;
using TileW32n16 = ConvTile<4, 32, 1, 8, 16>;

static void tile_dims(int t, int& th, int& tw, int& imgs, int& ck, int& bn) {
  switch (t) {
    case 0: th = 4; tw = 32; imgs = 1; ck = 8; break;
    case 1: th = 8; tw = 16; imgs = 1; ck = 8; break;
    case 2: th = 8; tw = 8; imgs = 2; ck = 8; break;
    case 3: th = 4; tw = 4; imgs = 8; ck = 8; break;
    case 4: th = 2; tw = 2; imgs = 32; ck = 8; break;
    case 5: th = 4; tw = 32; imgs = 1; ck = 4; break;
    default: th = 4; tw = 32; imgs = 1; ck = 8; bn = 16; return;
  }
  bn = 64;
}

static IgemmPlan igemm_plan(int N, int Cin, int H, int W, int Cout) {
  IgemmPlan p{};
  if (Cout <= 16 && Cin > 4 && W >= 32) p.tile = 6;
  else if (Cin <= 4 && W >= 32) p.tile = 5;
  else if (W >= 32) p.tile = 0;
  else if (W >= 16) p.tile = 1;
  else if (W >= 8) p.tile = 2;
  else if (W >= 4) p.tile = 3;
  else p.tile = 4;
  int th, tw, imgs, ck, bn;
  tile_dims(p.tile, th, tw, imgs, ck, bn);
  p.tiles_w = cdiv(W, tw);
  p.tiles_h = cdiv(H, th);
  p.tiles_n = cdiv(N, imgs);
  p.co_tiles = cdiv(Cout, bn);
  p.nchunks = cdiv(Cin, ck);
  long blocks = (long)p.tiles_w * p.tiles_h * p.tiles_n * p.co_tiles;
  const long target = 512;  // two resident blocks on each of 256 CUs
  int splits = 1;
  if (blocks < target) splits = (int)std::min<long>(p.nchunks, cdiv((int)target, (int)blocks));
  p.cps = cdiv(p.nchunks, splits);
  p.splits = cdiv(p.nchunks, p.cps);
  p.ws_bytes = p.splits > 1 ? (size_t)p.splits * N * Cout * H * W * sizeof(float) : 0;
  return p;
}

template <class T, bool DGRAD>
static void igemm_launch(const IgemmPlan& p, const float* in, const float* wt,
                         const float* bias, const float* mask, float* out, float* ws,
                         int N, int Cin, int H, int W, int Cout, int relu, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    hipFuncSetAttribute((const void*)conv3x3_igemm_f32<T, DGRAD>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
    attr_set = true;
  }
  dim3 grid(p.tiles_w * p.tiles_h * p.tiles_n, p.co_tiles, p.splits);
  const bool part = p.splits > 1;
  conv3x3_igemm_f32<T, DGRAD><<<grid, 256, T::LDS_BYTES, st>>>(
      in, wt, part ? nullptr : bias, part ? nullptr : mask, part ? ws : out, N, Cin, H, W,
      Cout, p.tiles_w, p.tiles_h, p.cps, part ? 0 : relu, part ? 1 : 0);
  if (part) {
    size_t total = (size_t)N * Cout * H * W;
    conv_splitk_reduce<<<(unsigned)((total + 63) / 64), 256, 0, st>>>(
        ws, p.splits, total, Cout, (size_t)H * W, bias, relu, mask, out);
  }
}

template <bool DGRAD>
static void igemm_dispatch(const IgemmPlan& p, const float* in, const float* wt,
                           const float* bias, const float* mask, float* out, float* ws,
                           int N, int Cin, int H, int W, int Cout, int relu, hipStream_t st) {
  switch (p.tile) {
    case 0: igemm_launch<TileW32, DGRAD>(p, in, wt, bias, mask, out, ws, N, Cin, H, W, Cout, relu, st); break;
    case 1: igemm_launch<TileW16, DGRAD>(p, in, wt, bias, mask, out, ws, N, Cin, H, W, Cout, relu, st); break;
    case 2: igemm_launch<TileW8, DGRAD>(p, in, wt, bias, mask, out, ws, N, Cin, H, W, Cout, relu, st); break;
    case 3: igemm_launch<TileW4, DGRAD>(p, in, wt, bias, mask, out, ws, N, Cin, H, W, Cout, relu, st); break;
    case 4: igemm_launch<TileW2, DGRAD>(p, in, wt, bias, mask, out, ws, N, Cin, H, W, Cout, relu, st); break;
    case 5: igemm_launch<TileW32c4, DGRAD>(p, in, wt, bias, mask, out, ws, N, Cin, H, W, Cout, relu, st); break;
    default: igemm_launch<TileW32n16, DGRAD>(p, in, wt, bias, mask, out, ws, N, Cin, H, W, Cout, relu, st); break;
  }
}

}  // namespace sb

// Entry points used by api.hip.
namespace sbh {

size_t conv_igemm_ws(int N, int Cin, int H, int W, int Cout) {
  return sb::igemm_plan(N, Cin, H, W, Cout).ws_bytes;
}

int conv_igemm_describe(bool dgrad, int N, int Cin, int H, int W, int Cout, char* buf,
                        size_t len) {
  sb::IgemmPlan p = sb::igemm_plan(N, Cin, H, W, Cout);
  int th, tw, imgs, ck, bn;
  sb::tile_dims(p.tile, th, tw, imgs, ck, bn);
  return snprintf(buf, len,
                  "sb::conv3x3_igemm_f32<sb::ConvTile<%d, %d, %d, %d, %d>, %s> grid=%dx%dx%d%s",
                  th, tw, imgs, ck, bn, dgrad ? "true" : "false",
                  p.tiles_w * p.tiles_h * p.tiles_n, p.co_tiles, p.splits,
                  p.splits > 1 ? " +sb::conv_splitk_reduce" : "");
}

sb_status conv_igemm_f32(bool dgrad, int N, int Cin, int H, int W, int Cout, const float* in,
                         const float* wt, const float* bias, const float* mask, float* out,
                         void* ws, size_t ws_bytes, int relu, hipStream_t st) {
  sb::IgemmPlan p = sb::igemm_plan(N, Cin, H, W, Cout);
  if (p.ws_bytes > 0 && (ws == nullptr || ws_bytes < p.ws_bytes)) return SB_ERR_WORKSPACE;
  if (dgrad)
    sb::igemm_dispatch<true>(p, in, wt, bias, mask, out, (float*)ws, N, Cin, H, W, Cout, relu, st);
  else
    sb::igemm_dispatch<false>(p, in, wt, bias, mask, out, (float*)ws, N, Cin, H, W, Cout, relu, st);
  return launch_status();
}

}  // namespace sbh
