// conv_wgrad.hip -- 3x3 / stride 1 / pad 1 convolution weight and bias
// gradients on fp32 MFMA (sec. 2.2 backward propagation):
//   dw[k,c,r,s] = sum_{n,h,w} x[n,c,h+r-1,w+s-1] * dy[n,k,h,w]
//   db[k]       = sum_{n,h,w} dy[n,k,h,w]
//
// GEMM view: rows = output channels k, columns = (input channel c, tap),
// reduction = every pixel of the batch.  A block owns 64 k and walks a
// contiguous range of 64-pixel tiles (IMGS images x TH rows x TW cols).  Per
// pixel tile it stages in LDS
//   * dy: 64 k x 64 pixels, stored [pixel][k] so an MFMA operand read of 16
//     consecutive k is bank-conflict free, and
//   * the x halo: BC channels x IMGS x (TH+2) x (TW+2), stored [halo pixel][c],
//     read once and shifted per tap.
// Two column layouts:
//   * wide (C >= 16): a block owns 16 channels x 9 taps; per 4-pixel step a
//     wave multiplies one dy fragment against 9 tap-shifted x fragments.
//   * narrow (C <= 7, e.g. the RGB input layer): a block owns every (c, tap)
//     pair, flattened into NCB blocks of 16 MFMA columns; each lane gathers
//     its own (c, tap) from the halo, so only the padding of C*9 up to a
//     multiple of 16 is wasted instead of 16 - C channels.
// Blocks of the first column tile also multiply dy against a column of ones,
// which yields the bias gradient in the same pass.
//
// The reduction dimension is long (up to N*H*W = 131072 here) while the
// output is small, so pixel tiles are split over gridDim.z; each split writes
// its partial sums to the workspace and splits_reduce adds the splits in a
// fixed order.  No atomics: results are bitwise reproducible.
#include "sb_internal.hpp"

#include <algorithm>
#include <cstdio>

namespace sb {

template <int TH_, int TW_, int IMGS_, int NCB_>
struct WgTile {
  static constexpr int TH = TH_, TW = TW_, IMGS = IMGS_;
  static constexpr int NCB = NCB_;                  // 0: wide layout; else narrow column blocks
  static constexpr bool NARROW = NCB_ > 0;
  static constexpr int BP = IMGS * TH * TW;         // pixels per tile
  static_assert(BP == 64, "64-pixel tiles");
  static_assert(TW % 4 == 0 || (TW == 2 && TH == 2), "4-pixel steps must map uniformly");
  static constexpr int BK = 64;
  static constexpr int BC = NARROW ? 8 : 16;        // channels staged per block
  static constexpr int NACC = NARROW ? NCB : 9;     // accumulator blocks per wave
  static constexpr int HH = TH + 2, HW = TW + 2;
  static constexpr int PLANE = IMGS * HH * HW;      // halo pixels per channel
  static constexpr int DY_STRIDE = BK + 16;         // floats per pixel row of dy
  static constexpr int LDS_DY = BP * DY_STRIDE;
  static constexpr int LDS_X = PLANE * BC;
  static constexpr int LDS_BUF = LDS_DY + LDS_X;
  static constexpr int DY_PT = BK * BP / 256;       // 16
  static constexpr int X_PT = (BC * PLANE + 255) / 256;
  static constexpr size_t LDS_BYTES = 2 * LDS_BUF * sizeof(float);
};

// Halo offset of tile pixel p (0..BP-1).
template <class T>
__device__ __forceinline__ int wg_hoff(int p) {
  int img = p / (T::TH * T::TW), r = p - img * (T::TH * T::TW);
  int yy = r / T::TW, xx = r - yy * T::TW;
  return img * T::HH * T::HW + yy * T::HW + xx;
}

template <class T>
__global__ __launch_bounds__(256, 2) void conv3x3_wgrad_f32(
    const float* __restrict__ x, const float* __restrict__ dy, float* __restrict__ dw,
    float* __restrict__ db, int N, int C, int H, int W, int K, int tiles_w, int tiles_h,
    int ptiles, int tiles_per_split, int c_tiles, int partial) {
  extern __shared__ float lds[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int jq = lane >> 4, lr = lane & 15;
  const int ct = blockIdx.x % c_tiles, kt = blockIdx.x / c_tiles;
  const int c0 = ct * T::BC, k0 = kt * T::BK;
  const int pt0 = blockIdx.z * tiles_per_split;
  const int pt1 = min(ptiles, pt0 + tiles_per_split);
  const bool do_db = (db != nullptr) && ct == 0;
  const size_t HWs = (size_t)H * W;

  // Lane offset of pixel (step base + jq) relative to the step base's halo offset.
  const int lane_hoff = wg_hoff<T>(jq);

  // Narrow layout: this lane's (c, tap) column in each column block.
  int col_off[T::NARROW ? T::NCB : 1];
  bool col_ok[T::NARROW ? T::NCB : 1];
  if (T::NARROW) {
#pragma unroll
    for (int cb = 0; cb < (T::NARROW ? T::NCB : 1); ++cb) {
      int j = cb * 16 + lr, c = j / 9, t = j - c * 9;
      col_ok[cb] = j < C * 9;
      col_off[cb] = col_ok[cb] ? ((t / 3) * T::HW + (t % 3)) * T::BC + c : 0;
    }
  }

  f4 acc[T::NACC], accb = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < T::NACC; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};

  float rdy[T::DY_PT], rx[T::X_PT];

  auto tile_origin = [&](int pt, int& n0, int& h0, int& w0) {
    int tx = pt % tiles_w, r = pt / tiles_w;
    int ty = r % tiles_h, tn = r / tiles_h;
    n0 = tn * T::IMGS; h0 = ty * T::TH; w0 = tx * T::TW;
  };

  auto gload = [&](int pt) {
    int n0, h0, w0;
    tile_origin(pt, n0, h0, w0);
    // dy: element e = (k-in-tile, pixel) with pixel fastest (coalesced rows).
#pragma unroll
    for (int i = 0; i < T::DY_PT; ++i) {
      int e = tid + i * 256;
      int kk = e / T::BP, p = e - kk * T::BP;
      int img = p / (T::TH * T::TW), r = p - img * (T::TH * T::TW);
      int yy = r / T::TW, xx = r - yy * T::TW;
      int n = n0 + img, h = h0 + yy, w = w0 + xx, k = k0 + kk;
      bool ok = n < N && h < H && w < W && k < K;
      rdy[i] = ok ? dy[((size_t)n * K + k) * HWs + (size_t)h * W + w] : 0.f;
    }
    // x halo: element e = (c-in-tile, halo pixel) with halo pixel fastest.
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) {
      int e = tid + i * 256;
      int cc = e / T::PLANE, hp = e - cc * T::PLANE;
      int img = hp / (T::HH * T::HW), r = hp - img * (T::HH * T::HW);
      int yy = r / T::HW, xx = r - yy * T::HW;
      int n = n0 + img, h = h0 + yy - 1, w = w0 + xx - 1, c = c0 + cc;
      bool ok = e < T::BC * T::PLANE && n < N && h >= 0 && h < H && w >= 0 && w < W && c < C;
      rx[i] = ok ? x[((size_t)n * C + c) * HWs + (size_t)h * W + w] : 0.f;
    }
  };
  auto lstore = [&](int buf) {
    float* Dl = lds + buf * T::LDS_BUF;
    float* Xl = Dl + T::LDS_DY;
#pragma unroll
    for (int i = 0; i < T::DY_PT; ++i) {
      int e = tid + i * 256;
      int kk = e / T::BP, p = e - kk * T::BP;
      Dl[p * T::DY_STRIDE + kk] = rdy[i];
    }
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) {
      int e = tid + i * 256;
      if (e < T::BC * T::PLANE) {
        int cc = e / T::PLANE, hp = e - cc * T::PLANE;
        Xl[hp * T::BC + cc] = rx[i];
      }
    }
  };

  if (pt0 < pt1) {
    gload(pt0);
    lstore(0);
  }
  __syncthreads();

  for (int pt = pt0; pt < pt1; ++pt) {
    const int buf = (pt - pt0) & 1;
    const bool more = pt + 1 < pt1;
    if (more) gload(pt + 1);
    const float* Dl = lds + buf * T::LDS_BUF;
    const float* Xl = Dl + T::LDS_DY;
#pragma unroll
    for (int st = 0; st < T::BP / 4; ++st) {
      const int pbase = st * 4;
      const int hbase = wg_hoff<T>(pbase);          // compile-time after unrolling
      float a = Dl[(pbase + jq) * T::DY_STRIDE + wave * 16 + lr];
      const float* Xp = Xl + (hbase + lane_hoff) * T::BC;
      if (T::NARROW) {
#pragma unroll
        for (int cb = 0; cb < T::NACC; ++cb) {
          float b = Xp[col_off[cb % (T::NARROW ? T::NCB : 1)]];
          b = col_ok[cb % (T::NARROW ? T::NCB : 1)] ? b : 0.f;
          acc[cb] = mfma16x16x4(a, b, acc[cb]);
        }
      } else {
#pragma unroll
        for (int t = 0; t < 9; ++t) {
          const int toff = (t / 3) * T::HW + (t % 3);
          float b = Xp[toff * T::BC + lr];
          acc[t] = mfma16x16x4(a, b, acc[t]);
        }
      }
      if (do_db) accb = mfma16x16x4(a, 1.0f, accb);
    }
    if (more) lstore(buf ^ 1);
    __syncthreads();
  }

  // acc[t] lane holds rows k = k0 + wave*16 + 4*jq + i and column lr of its block.
  const size_t wsz = (size_t)K * C * 9;
  float* dst = dw + (partial ? (size_t)blockIdx.z * wsz : 0);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int k = k0 + wave * 16 + 4 * jq + i;
    if (k >= K) continue;
    if (T::NARROW) {
#pragma unroll
      for (int cb = 0; cb < T::NACC; ++cb) {
        int j = cb * 16 + lr;                       // flattened (c, tap)
        if (j < C * 9) dst[(size_t)k * C * 9 + j] = acc[cb][i];
      }
    } else {
      int c = c0 + lr;
      if (c >= C) continue;
#pragma unroll
      for (int t = 0; t < 9; ++t) dst[((size_t)k * C + c) * 9 + t] = acc[t][i];
    }
  }
  if (do_db && lr == 0) {
    float* dbd = db + (partial ? (size_t)blockIdx.z * K : 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int k = k0 + wave * 16 + 4 * jq + i;
      if (k < K) dbd[k] = accb[i];
    }
  }
}

// dst[i] = sum over the splits of part[s*total + i], in a fixed order.
__global__ __launch_bounds__(256) void splits_reduce(const float* __restrict__ part, int splits,
                                                     size_t total, float* __restrict__ dst) {
  __shared__ float lds[256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t i = (size_t)blockIdx.x * 64 + lane;
  float v = SplitSum{part, splits, total}(i, wave, lds, lane);
  if (wave == 0 && i < total) dst[i] = v;
}

struct WgPlan {
  int tile, tiles_w, tiles_h, ptiles, k_tiles, c_tiles, tps, splits;
  size_t ws_bytes;
};

// Wide layouts (16 channels x 9 taps per block), by image width.
using WgW32 = WgTile<2, 32, 1, 0>;
using WgW16 = WgTile<4, 16, 1, 0>;
using WgW8 = WgTile<8, 8, 1, 0>;
using WgW4 = WgTile<4, 4, 4, 0>;
using WgW2 = WgTile<2, 2, 16, 0>;
// Narrow layouts (all C <= 7 channels x 9 taps in NCB column blocks).
using WgN32_2 = WgTile<2, 32, 1, 2>;   // C <= 3
using WgN32_4 = WgTile<2, 32, 1, 4>;   // C <= 7
using WgN4_2 = WgTile<4, 4, 4, 2>;
using WgN4_4 = WgTile<4, 4, 4, 4>;

static WgPlan wg_plan(int N, int C, int H, int W, int K) {
  WgPlan p{};
  int th, tw, imgs;
  const bool narrow = C <= 7;
  if (narrow) {
    // 32-wide rows for wide images, 4x4 x 4-image tiles otherwise.
    if (W >= 32) { th = 2; tw = 32; imgs = 1; p.tile = C <= 3 ? 5 : 6; }
    else { th = 4; tw = 4; imgs = 4; p.tile = C <= 3 ? 7 : 8; }
  } else if (W >= 32) { p.tile = 0; th = 2; tw = 32; imgs = 1; }
  else if (W >= 16) { p.tile = 1; th = 4; tw = 16; imgs = 1; }
  else if (W >= 8) { p.tile = 2; th = 8; tw = 8; imgs = 1; }
  else if (W >= 4) { p.tile = 3; th = 4; tw = 4; imgs = 4; }
  else { p.tile = 4; th = 2; tw = 2; imgs = 16; }
  p.tiles_w = cdiv(W, tw);
  p.tiles_h = cdiv(H, th);
  p.ptiles = p.tiles_w * p.tiles_h * cdiv(N, imgs);
  p.k_tiles = cdiv(K, 64);
  p.c_tiles = narrow ? 1 : cdiv(C, 16);
  long blocks = (long)p.k_tiles * p.c_tiles;
  // About two blocks per CU, but at most 128 splits of the pixel range.
  const long target = 512;
  int splits = 1;
  if (blocks < target)
    splits = (int)std::min<long>(std::min<long>(p.ptiles, 128), cdiv((int)target, (int)blocks));
  p.tps = cdiv(p.ptiles, splits);
  p.splits = cdiv(p.ptiles, p.tps);
  p.ws_bytes = p.splits > 1 ? (size_t)p.splits * ((size_t)K * C * 9 + K) * sizeof(float) : 0;
  return p;
}

template <class T>
static void wg_launch(const WgPlan& p, const float* x, const float* dy, float* dw, float* db,
                      float* ws, int N, int C, int H, int W, int K, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    hipFuncSetAttribute((const void*)conv3x3_wgrad_f32<T>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
    attr_set = true;
  }
  dim3 grid(p.k_tiles * p.c_tiles, 1, p.splits);
  const bool part = p.splits > 1;
  const size_t wsz = (size_t)K * C * 9;
  float* pdw = part ? ws : dw;
  float* pdb = db ? (part ? ws + (size_t)p.splits * wsz : db) : nullptr;
  conv3x3_wgrad_f32<T><<<grid, 256, T::LDS_BYTES, st>>>(
      x, dy, pdw, pdb, N, C, H, W, K, p.tiles_w, p.tiles_h, p.ptiles, p.tps, p.c_tiles,
      part ? 1 : 0);
  if (part) {
    splits_reduce<<<(unsigned)((wsz + 63) / 64), 256, 0, st>>>(ws, p.splits, wsz, dw);
    if (db)
      splits_reduce<<<(unsigned)((K + 63) / 64), 256, 0, st>>>(pdb, p.splits, (size_t)K, db);
  }
}

}  // namespace sb

namespace sbh {

size_t conv_wgrad_ws(int N, int C, int H, int W, int K) {
  return sb::wg_plan(N, C, H, W, K).ws_bytes;
}

int conv_wgrad_describe(int N, int C, int H, int W, int K, char* buf, size_t len) {
  static const char* names[] = {"2, 32, 1, 0", "4, 16, 1, 0", "8, 8, 1, 0", "4, 4, 4, 0",
                                "2, 2, 16, 0", "2, 32, 1, 2", "2, 32, 1, 4", "4, 4, 4, 2",
                                "4, 4, 4, 4"};
  sb::WgPlan p = sb::wg_plan(N, C, H, W, K);
  return snprintf(buf, len, "sb::conv3x3_wgrad_f32<sb::WgTile<%s> > grid=%dx1x%d%s",
                  names[p.tile], p.k_tiles * p.c_tiles, p.splits,
                  p.splits > 1 ? " +sb::splits_reduce" : "");
}

sb_status conv_wgrad_f32(int N, int C, int H, int W, int K, const float* x, const float* dy,
                         float* dw, float* db, void* ws, size_t ws_bytes, hipStream_t st) {
  sb::WgPlan p = sb::wg_plan(N, C, H, W, K);
  if (p.ws_bytes > 0 && (ws == nullptr || ws_bytes < p.ws_bytes)) return SB_ERR_WORKSPACE;
  float* w = (float*)ws;
  switch (p.tile) {
    case 0: sb::wg_launch<sb::WgW32>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
    case 1: sb::wg_launch<sb::WgW16>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
    case 2: sb::wg_launch<sb::WgW8>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
    case 3: sb::wg_launch<sb::WgW4>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
    case 4: sb::wg_launch<sb::WgW2>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
    case 5: sb::wg_launch<sb::WgN32_2>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
    case 6: sb::wg_launch<sb::WgN32_4>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
    case 7: sb::wg_launch<sb::WgN4_2>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
    default: sb::wg_launch<sb::WgN4_4>(p, x, dy, dw, db, w, N, C, H, W, K, st); break;
  }
  return launch_status();
}

}  // namespace sbh
