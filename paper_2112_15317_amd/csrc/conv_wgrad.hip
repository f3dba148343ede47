// conv_wgrad.hip -- 3x3 / stride 1 / pad 1 convolution weight and bias
// gradients on fp32 MFMA (sec. 2.2 backward propagation):
//   dw[k,c,r,s] = sum_{n,h,w} x[n,c,h+r-1,w+s-1] * dy[n,k,h,w]
//   db[k]       = sum_{n,h,w} dy[n,k,h,w]
//
// GEMM view: rows = output channels k, columns = (input channel c, tap),
// reduction = every pixel of the batch.  The bias gradient comes in the same
// pass: each lane adds up the dy operands it feeds the MFMAs on the vector
// ALU (which runs beside the matrix pipe), and a butterfly over the lanes
// completes the row sums; only blocks of the first column tile write them.
// An MFMA against a column of ones in those blocks alone would make them
// the slowest of the grid.  Three kernels:
//
// conv3x3_wgrad_f32 (any shape).  A block owns 64 k and walks a contiguous
// range of 64-pixel tiles (IMGS images x TH rows x TW cols).  Per pixel tile
// it stages in LDS dy (64 k x 64 pixels, stored [pixel][k] so an operand
// read of 16 consecutive k is conflict-free) and the x halo (BC channels x
// IMGS x (TH+2) x (TW+2), stored [halo pixel][c], shifted per tap).  Column
// layouts:
//   * wide (C >= 8): a block owns 16 channels x 9 taps; per 4-pixel step a
//     wave multiplies one dy fragment against 9 tap-shifted x fragments.
//   * narrow (C <= 7, e.g. the RGB input layer): a block owns every (c, tap)
//     pair, flattened into NCB blocks of 16 MFMA columns; each lane gathers
//     its own (c, tap), so only C*9 rounded up to 16 is computed.
//
// conv3x3_wgrad_2x2 (2x2 images): every (output, input) position pair of
// an image is a tap inside it, so the gradient is one dense GEMM over the
// images with rows (k, position) and columns (c, position), folded into the
// 9 taps in the epilogue.
//
// conv3x3_wgrad_small_f32 (whole images of 4x4 pixels).  The
// reduction runs over 4 images at a time at one pixel position; for each
// (position, tap) pair whose source lies inside the image (known at compile
// time) one MFMA adds dy[., k, pos] x x[., c, src(pos, tap)] into tap's
// accumulator.  Padded taps are never multiplied.  LDS holds dy as
// [position][image][k] and x as [position][image][c], filled with float4
// loads of whole image planes.
//
// The reduction dimension is long (up to N*H*W = 131072) while the output is
// small, so the pixels are split over gridDim.z; each split writes its
// partial sums to the workspace and splits_reduce adds the splits in a fixed
// order.  No float atomics: results are bitwise reproducible.
#include "sb_internal.hpp"

#include <algorithm>
#include <cstdio>
#include <mutex>

namespace sb {

struct WgArgs {
  const void* x;         // [N][C][H][W], element type E of the kernel
  const void* dy;        // [N][K][H][W], element type E
  float* dw;             // [K][C][3][3]
  float* db;             // [K] or null
  float* part;           // split partials: [splits][K*C*9 + K] (dw, then db)
  int N, C, H, W, K;
  int tiles_w, tiles_h, ptiles, tiles_per_split, c_tiles, splits;
};

// Buffer resource over `imgs` images (clipped to the batch) of an NCHW tensor
// from image n0 on; per_img = elements per image.
template <class E>
__device__ __forceinline__ rsrc_t image_rsrc(const void* t, int n0, int imgs, int N, int per_img) {
  const int cnt = min(imgs, N - n0);
  return make_rsrc((const E*)t + (size_t)n0 * per_img,
                   (uint32_t)((size_t)cnt * per_img * sizeof(E)));
}

// The block's (column block, split) = (x, z), with the hardware block ids
// remapped so that each of the 8 XCDs runs whole splits: the dispatcher
// deals consecutive blocks round-robin to the XCDs, and all column blocks
// of a split read the same pixel tiles of x and dy, which then come from
// that XCD's L2 instead of every XCD fetching them.  Grids whose size is
// not a multiple of 8 keep the plain order.
struct WgBlock { int x, z; };
__device__ __forceinline__ WgBlock wg_block() {
  const int gx = gridDim.x, nb = gx * gridDim.z;
  int h = blockIdx.x + gx * blockIdx.z;
  if (nb % 8 == 0) h = (h % 8) * (nb / 8) + h / 8;
  return WgBlock{h % gx, h / gx};
}

// Writes (or split-reduces) the block's 64 k x 16-column x NACC outputs.
// `val(i, t)` is the lane's accumulator t, element i; `col(t)` the flattened
// (c, tap) column of the lane in accumulator t, or -1.
template <int NACC, class Val, class Col>
__device__ __forceinline__ void wgrad_store(const WgArgs& a, int z, int k_base, bool do_db,
                                            const f4& accb, Val val, Col col) {
  const int lane = threadIdx.x & 63, jq = lane >> 4, lr = lane & 15;
  const size_t wsz = (size_t)a.K * a.C * 9;
  auto each = [&](auto&& fn) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = k_base + 4 * jq + i;
      if (k >= a.K) continue;
#pragma unroll
      for (int t = 0; t < NACC; ++t) {
        const int j = col(t);
        if (j >= 0) fn(val(i, t), (size_t)k * a.C * 9 + j);
      }
    }
  };
  auto each_db = [&](auto&& fn) {
    if (!do_db || lr != 0) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = k_base + 4 * jq + i;
      if (k < a.K) fn(accb[i], k);
    }
  };
  if (a.splits == 1) {
    each([&](float v, size_t o) { a.dw[o] = v; });
    each_db([&](float v, int k) { a.db[k] = v; });
    return;
  }
  float* pw = a.part + (size_t)z * (wsz + a.K);
  float* pb = pw + wsz;
  each([&](float v, size_t o) { pw[o] = v; });
  each_db([&](float v, int k) { pb[k] = v; });
}

// Sum over the splits of part[s*stride + i], in a fixed order, for i < count:
// dw[i] for i < wsz, then db[i - wsz].
__global__ __launch_bounds__(256) void splits_reduce(const float* __restrict__ part, int splits,
                                                     size_t stride, size_t count, size_t wsz,
                                                     float* __restrict__ dw,
                                                     float* __restrict__ db) {
  __shared__ float lds[256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t i = (size_t)blockIdx.x * 64 + lane;
  float v = SplitSum{part, splits, stride, count}(i, wave, lds, lane);
  if (wave != 0 || i >= count) return;
  if (i < wsz) dw[i] = v;
  else db[i - wsz] = v;
}

// The same for 4 consecutive outputs per thread (stride and count multiples
// of 4): all splits of a thread's outputs summed in one thread, in order.
__global__ __launch_bounds__(256) void splits_reduce4(const float* __restrict__ part, int splits,
                                                      size_t stride, size_t count, size_t wsz,
                                                      float* __restrict__ dw,
                                                      float* __restrict__ db) {
  const size_t i4 = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i4 >= count) return;
  const f4 v = split_sum4(part, splits, stride, i4);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const size_t i = i4 + j;
    if (i < wsz) dw[i] = v[j];
    else db[i - wsz] = v[j];
  }
}

// The same with the splits shared out over the G waves of a block: wave w
// sums its contiguous range of splits in order, then the G range sums are
// added in wave order (fixed for a given shape, so still deterministic).
template <int G>
__global__ __launch_bounds__(64 * G) void splits_reduce4w(const float* __restrict__ part,
                                                          int splits, size_t stride,
                                                          size_t count, size_t wsz,
                                                          float* __restrict__ dw,
                                                          float* __restrict__ db) {
  __shared__ f4 red[G][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t i4 = ((size_t)blockIdx.x * 64 + lane) * 4;
  const int per = (splits + G - 1) / G;
  const int s0 = min(splits, wave * per), s1 = min(splits, s0 + per);
  red[wave][lane] = i4 < count ? split_sum4(part, s0, s1, stride, i4) : f4{0.f, 0.f, 0.f, 0.f};
  __syncthreads();
  if (wave != 0 || i4 >= count) return;
  f4 v = red[0][lane];
#pragma unroll
  for (int w = 1; w < G; ++w) v += red[w][lane];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const size_t i = i4 + j;
    if (i < wsz) dw[i] = v[j];
    else db[i - wsz] = v[j];
  }
}

// Launches the weight-gradient split reduction: dw (K*C*9) then, when db is
// wanted, db (K), from partials [splits][K*C*9 + K].
inline void launch_splits_reduce(const float* part, int splits, int K, int C, float* dw,
                                 float* db, hipStream_t st) {
  const size_t wsz = (size_t)K * C * 9, stride = wsz + K;
  const size_t count = wsz + (db ? K : 0);
  if (stride % 4 == 0 && count % 4 == 0 && ((uintptr_t)part & 15) == 0) {
    const unsigned blocks64 = (unsigned)((count / 4 + 63) / 64);
    switch (split_waves(count, splits)) {
      case 1:
        splits_reduce4<<<(unsigned)((count / 4 + 255) / 256), 256, 0, st>>>(
            part, splits, stride, count, wsz, dw, db);
        break;
      case 2:
        splits_reduce4w<2><<<blocks64, 128, 0, st>>>(part, splits, stride, count, wsz, dw, db);
        break;
      case 4:
        splits_reduce4w<4><<<blocks64, 256, 0, st>>>(part, splits, stride, count, wsz, dw, db);
        break;
      case 8:
        splits_reduce4w<8><<<blocks64, 512, 0, st>>>(part, splits, stride, count, wsz, dw, db);
        break;
      default:
        splits_reduce4w<16><<<blocks64, 1024, 0, st>>>(part, splits, stride, count, wsz, dw, db);
        break;
    }
  } else
    splits_reduce<<<(unsigned)((count + 63) / 64), 256, 0, st>>>(part, splits, stride, count,
                                                                wsz, dw, db);
}

// Bias gradient of a wave's 16 rows, summed on the vector ALU beside the
// MFMAs: lane (jq, lr) has added the dy values it supplied as MFMA operand
// (row lr, the pixels of lane group jq).  Returns the row sums in the MFMA
// result layout the stores expect: element i of lane (jq, lr) is row
// 4 jq + i.  A fixed butterfly: bitwise reproducible.
__device__ __forceinline__ f4 wave_row_sums(float s) {
  s += __shfl_xor(s, 16, 64);
  s += __shfl_xor(s, 32, 64);
  const int jq = (threadIdx.x & 63) >> 4;
  return f4{__shfl(s, 4 * jq + 0, 64), __shfl(s, 4 * jq + 1, 64), __shfl(s, 4 * jq + 2, 64),
            __shfl(s, 4 * jq + 3, 64)};
}

// Writes a block's weight gradient of 64 k x (16 c x 9 taps): acc[t] of wave
// w, lane (jq, lr) holds rows k0 + 16 w + 4 jq + i, channel c0 + lr, tap t.
// The tile goes out through LDS (64 x 148 floats, free when this is called)
// as 64 rows of 144 consecutive floats (k, then c * 9 + tap: the dw order),
// written in 16-byte pieces, to dw or to this split's partials; otherwise
// each lane would write single floats 9 apart.
__device__ __forceinline__ void wgrad_store_rows(const WgArgs& a, int z, int k0, int c0,
                                                 bool do_db, const f4& accb, const f4 (&acc)[9],
                                                 float* lds) {
  constexpr int BK = 64, RW = 16 * 9, RP = RW + 4, QPR = RW / 4;
  const int tid = threadIdx.x, wave = tid >> 6, jq = (tid & 63) >> 4, lr = tid & 15;
  const int cw = min(16, a.C - c0) * 9;              // live columns of the tile
  const size_t wsz = (size_t)a.K * a.C * 9;
  float* dst = a.splits == 1 ? a.dw : a.part + (size_t)z * (wsz + a.K);
  const bool vec = (a.C * 9) % 4 == 0 && cw % 4 == 0 &&
                   (((uintptr_t)dst + (size_t)c0 * 9 * sizeof(float)) & 15) == 0;
#pragma unroll
  for (int t = 0; t < 9; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) lds[(wave * 16 + 4 * jq + i) * RP + lr * 9 + t] = acc[t][i];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < BK * QPR / 256; ++j) {
    const int q = tid + 256 * j, row = q / QPR, col = (q % QPR) * 4, k = k0 + row;
    if (k >= a.K || col >= cw) continue;
    float* o = dst + (size_t)k * a.C * 9 + (size_t)c0 * 9 + col;
    const float* l = lds + row * RP + col;
    if (vec) {
      *reinterpret_cast<f4*>(o) = *reinterpret_cast<const f4*>(l);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (col + e < cw) o[e] = l[e];
    }
  }
  if (do_db && lr == 0) {
    float* pb = a.splits == 1 ? a.db : dst + wsz;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = k0 + wave * 16 + 4 * jq + i;
      if (k < a.K) pb[k] = accb[i];
    }
  }
}

// ----------------------------------------------------------------- generic --
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
  // dy tile [k][pixel], rows 68 floats apart (4 mod 64 banks): the 16 rows
  // x 4 pixels of an operand read and of a staging write hit 64 banks.
  static constexpr int DYP = BP + 4;
  static constexpr int LDS_DY = BK * DYP;
  static constexpr int LDS_X = PLANE * BC;
  static constexpr int LDS_BUF = LDS_DY + LDS_X;
  static constexpr int DY_PT = BK * BP / 256;       // 16
  static constexpr int X_PT = (BC * PLANE + 255) / 256;
  static constexpr size_t LDS_BYTES = 2 * LDS_BUF * sizeof(float);
  static_assert(LDS_BYTES <= 80 * 1024, "two blocks must fit in the 160 KB of LDS");
};

// Halo offset of tile pixel p (0..BP-1).
template <class T>
__device__ __forceinline__ int wg_hoff(int p) {
  int img = p / (T::TH * T::TW), r = p - img * (T::TH * T::TW);
  int yy = r / T::TW, xx = r - yy * T::TW;
  return img * T::HH * T::HW + yy * T::HW + xx;
}

// Whether the MFMA of 4-pixel step st at tap t only multiplies zero padding
// when a tile is one whole image (H = TH, W = TW): the step's pixels share a
// row, and a tap in the top (bottom) filter row reads the padding row above
// (below) the image for the image's first (last) row.  Known at compile time
// after unrolling, so those MFMAs are never issued.
template <class T, bool WHOLE>
__device__ constexpr bool wg_pad_step(int st, int t) {
  if (!WHOLE) return false;
  const int yy = (st * 4) % (T::TH * T::TW) / T::TW;
  return (t / 3 == 0 && yy == 0) || (t / 3 == 2 && yy == T::TH - 1);
}

// ROWS: every tile spans the image's full width (IMGS = 1, W = TW), so a
// staged element's offset within its image is a per-thread constant plus the
// tile's first row, and only its row can leave the image: the constants are
// worked out once per thread, and per tile an element costs an add and a row
// test.  WHOLE (with ROWS): every tile is a whole image (H = TH as well), and
// the steps whose taps read only padding are skipped (wg_pad_step).
// The block's work for block (x, z) of the layer `a`; the kernels below
// pick the layer and the block.
template <class T, class E, bool ROWS, bool WHOLE>
__device__ __forceinline__ void wgrad_f32_block(const WgArgs& a, const WgBlock blk) {
  static_assert(!WHOLE || (ROWS && T::IMGS == 1 && !T::NARROW), "whole-image tiles are full-width");
  extern __shared__ float lds[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int jq = lane >> 4, lr = lane & 15;
  const int ct = blk.x % a.c_tiles, kt = blk.x / a.c_tiles;
  const int c0 = ct * T::BC, k0 = kt * T::BK;
  const int pt0 = blk.z * a.tiles_per_split;
  const int pt1 = min(a.ptiles, pt0 + a.tiles_per_split);
  const bool do_db = (a.db != nullptr) && ct == 0;
  const int HWs = a.H * a.W;

  // Lane offset of pixel (step base + jq) relative to the step base's halo offset.
  const int lane_hoff = wg_hoff<T>(jq);

  // Narrow layout: this lane's (c, tap) column in each column block.
  constexpr int NC = T::NARROW ? T::NCB : 1;
  int col_off[NC];
  bool col_ok[NC];
#pragma unroll
  for (int cb = 0; cb < NC; ++cb) {
    int j = cb * 16 + lr, c = j / 9, t = j - c * 9;
    col_ok[cb] = T::NARROW && j < a.C * 9;
    col_off[cb] = col_ok[cb] ? ((t / 3) * T::HW + (t % 3)) * T::BC + c : 0;
  }

  f4 acc[T::NACC];
  float sbias = 0.f;     // this lane's share of its row's bias gradient
#pragma unroll
  for (int t = 0; t < T::NACC; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};

  float rdy[T::DY_PT], rx[T::X_PT];

  // Full-width tiles: each element's offset in its image for a tile at row
  // 0, and its row in the tile (dy) or halo (x); a row of kNone marks an
  // element that no tile has (k, channel or column outside, or past the
  // staged range).
  static_assert(!ROWS || T::IMGS == 1, "one image per full-width tile");
  constexpr int kNone = 1 << 20;
  int dy_rel[ROWS ? T::DY_PT : 1], dy_row[ROWS ? T::DY_PT : 1];
  int x_rel[ROWS ? T::X_PT : 1], x_row[ROWS ? T::X_PT : 1];
  if constexpr (ROWS) {
#pragma unroll
    for (int i = 0; i < T::DY_PT; ++i) {
      const int e = tid + i * 256;
      const int kk = (e >> 2) & (T::BK - 1), p = ((e >> 8) << 2) | (e & 3);
      const int yy = p / T::TW, xx = p % T::TW;
      dy_rel[i] = (k0 + kk) * HWs + yy * a.W + xx;
      dy_row[i] = k0 + kk < a.K ? yy : kNone;
    }
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) {
      const int e = tid + i * 256;
      const int hp = e / T::BC, cc = e - hp * T::BC;
      const int hy = hp / T::HW, w = hp % T::HW - 1, c = c0 + cc;
      const bool ok = e < T::BC * T::PLANE && c < a.C && (unsigned)w < (unsigned)a.W;
      x_rel[i] = c * HWs + (hy - 1) * a.W + w;
      x_row[i] = ok ? hy - 1 : kNone;
    }
  }

  auto gload = [&](int pt) {
    if constexpr (ROWS) {
      const int ty = pt % a.tiles_h, n0 = pt / a.tiles_h;
      const int h0 = ty * T::TH, hoff = h0 * a.W;
      const rsrc_t dr = image_rsrc<E>(a.dy, n0, 1, a.N, a.K * HWs);
      const rsrc_t xr = image_rsrc<E>(a.x, n0, 1, a.N, a.C * HWs);
#pragma unroll
      for (int i = 0; i < T::DY_PT; ++i)
        rdy[i] = BufLoad<E>::one(dr, h0 + dy_row[i] < a.H
                                         ? (uint32_t)(dy_rel[i] + hoff) * (uint32_t)sizeof(E)
                                         : kOOB);
#pragma unroll
      for (int i = 0; i < T::X_PT; ++i)
        rx[i] = BufLoad<E>::one(xr, (unsigned)(h0 + x_row[i]) < (unsigned)a.H
                                        ? (uint32_t)(x_rel[i] + hoff) * (uint32_t)sizeof(E)
                                        : kOOB);
      return;
    }
    int tx = pt % a.tiles_w, r0 = pt / a.tiles_w;
    int ty = r0 % a.tiles_h, tn = r0 / a.tiles_h;
    const int n0 = tn * T::IMGS, h0 = ty * T::TH, w0 = tx * T::TW;
    const rsrc_t dr = image_rsrc<E>(a.dy, n0, T::IMGS, a.N, a.K * HWs);
    const rsrc_t xr = image_rsrc<E>(a.x, n0, T::IMGS, a.N, a.C * HWs);
    // dy: element e = (pixel quad, k-in-tile, pixel within the quad).  A
    // wave covers 16 k x 4 consecutive pixels: 16 rows of 16 B in global
    // memory, and 64 distinct banks in the [k][pixel] LDS tile.
#pragma unroll
    for (int i = 0; i < T::DY_PT; ++i) {
      int e = tid + i * 256;
      int kk = (e >> 2) & (T::BK - 1), p = ((e >> 8) << 2) | (e & 3);
      int img = p / (T::TH * T::TW), r = p - img * (T::TH * T::TW);
      int yy = r / T::TW, xx = r - yy * T::TW;
      int n = n0 + img, h = h0 + yy, w = w0 + xx, k = k0 + kk;
      bool ok = n < a.N && h < a.H && w < a.W && k < a.K;
      const int off = (img * a.K + k) * HWs + h * a.W + w;          // from image n0
      rdy[i] = BufLoad<E>::one(dr, ok ? (uint32_t)off * (uint32_t)sizeof(E) : kOOB);
    }
    // x halo: element e = (halo pixel, c-in-tile) with c fastest, for the
    // same reason ([halo pixel][c] LDS tile).
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) {
      int e = tid + i * 256;
      int hp = e / T::BC, cc = e - hp * T::BC;
      int img = hp / (T::HH * T::HW), r = hp - img * (T::HH * T::HW);
      int yy = r / T::HW, xx = r - yy * T::HW;
      int n = n0 + img, h = h0 + yy - 1, w = w0 + xx - 1, c = c0 + cc;
      bool ok = e < T::BC * T::PLANE && n < a.N && h >= 0 && h < a.H && w >= 0 && w < a.W &&
                c < a.C;
      const int off = (img * a.C + c) * HWs + h * a.W + w;          // from image n0
      rx[i] = BufLoad<E>::one(xr, ok ? (uint32_t)off * (uint32_t)sizeof(E) : kOOB);
    }
  };
  auto lstore = [&](int buf) {
    float* Dl = lds + buf * T::LDS_BUF;
    float* Xl = Dl + T::LDS_DY;
#pragma unroll
    for (int i = 0; i < T::DY_PT; ++i) {
      int e = tid + i * 256;
      int kk = (e >> 2) & (T::BK - 1), p = ((e >> 8) << 2) | (e & 3);
      Dl[kk * T::DYP + p] = rdy[i];
    }
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) {
      int e = tid + i * 256;
      if (e < T::BC * T::PLANE) Xl[e] = rx[i];                 // = [halo pixel][c]
    }
  };
  // Operands of one 4-pixel step: the dy value and the NACC x values.  The
  // next step's operands are read from LDS before this step's MFMAs issue,
  // so their latency hides behind the MFMAs.
  struct Ops { float a, b[T::NACC]; };
  auto fetch = [&](const float* Dl, const float* Xl, int st) {
    Ops o;
    const int pbase = st * 4;
    const int hbase = wg_hoff<T>(pbase);            // compile-time after unrolling
    o.a = Dl[(wave * 16 + lr) * T::DYP + pbase + jq];
    const float* Xp = Xl + (hbase + lane_hoff) * T::BC;
    if (T::NARROW) {
#pragma unroll
      for (int cb = 0; cb < T::NACC; ++cb) {
        float b = Xp[col_off[cb % NC]];
        o.b[cb] = col_ok[cb % NC] ? b : 0.f;
      }
    } else {
#pragma unroll
      for (int t = 0; t < T::NACC; ++t) {
        const int toff = (t / 3) * T::HW + (t % 3);
        o.b[t] = wg_pad_step<T, WHOLE>(st, t) ? 0.f : Xp[toff * T::BC + lr];
      }
    }
    return o;
  };
  auto compute = [&](int buf) {
    const float* Dl = lds + buf * T::LDS_BUF;
    const float* Xl = Dl + T::LDS_DY;
    Ops cur = fetch(Dl, Xl, 0);
#pragma unroll
    for (int st = 0; st < T::BP / 4; ++st) {
      Ops nxt;
      if (st + 1 < T::BP / 4) nxt = fetch(Dl, Xl, st + 1);
#pragma unroll
      for (int t = 0; t < T::NACC; ++t)
        if (!wg_pad_step<T, WHOLE>(st, t)) acc[t] = mfma16x16x4(cur.a, cur.b[t], acc[t]);
      sbias += cur.a;
      if (st + 1 < T::BP / 4) cur = nxt;
    }
  };

  const int nt = pt1 - pt0;
  if (nt > 0) {
    gload(pt0);
    lstore(0);
    if (nt > 1) gload(pt0 + 1);
  }
  __syncthreads();
  for (int t = 0; t < nt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nt) lstore(buf ^ 1);
    if (t + 2 < nt) gload(pt0 + t + 2);
    compute(buf);
    __syncthreads();
  }

  const f4 accb = wave_row_sums(sbias);
  if constexpr (!T::NARROW) {
    static_assert(64 * (16 * 9 + 4) * sizeof(float) <= T::LDS_BYTES, "tile fits the LDS");
    wgrad_store_rows(a, blk.z, k0, c0, do_db, accb, acc, lds);
    return;
  }
  // acc[t] lane holds rows k = k0 + wave*16 + 4*jq + i and column lr of its block.
  wgrad_store<T::NACC>(
      a, blk.z, k0 + wave * 16, do_db, accb, [&](int i, int t) { return acc[t][i]; },
      [&](int t) -> int {
        if (T::NARROW) {
          int j = t * 16 + lr;
          return j < a.C * 9 ? j : -1;
        }
        int c = c0 + lr;
        return c < a.C ? c * 9 + t : -1;
      });
}

template <class T, class E, bool ROWS = false, bool WHOLE = false>
__global__ __launch_bounds__(256, 2) void conv3x3_wgrad_f32(WgArgs a) {
  wgrad_f32_block<T, E, ROWS, WHOLE>(a, wg_block());
}

// Weight gradients of up to kWgMany layers that take the same kernel, in
// one launch: layer i owns the blocks first[i] .. first[i+1]-1 of a 1-D
// grid, numbered within the layer as wg_block numbers a layer's own grid
// (dealt to the XCDs in whole splits when its block count and its first
// block are multiples of 8).  One launch instead of one per layer lets the
// next layer's blocks start while the previous layer's last blocks drain.
constexpr int kWgMany = 4;
struct WgMany {
  WgArgs a[kWgMany];
  int first[kWgMany + 1];   // first block of each layer, then the total
  int gx[kWgMany];          // the layer's column blocks (its grid's x extent)
  int n;
};

template <class T, class E, bool ROWS, bool WHOLE>
__global__ __launch_bounds__(256, 2) void conv3x3_wgrad_f32_many(WgMany m) {
  const int b = blockIdx.x;
  int i = 0;
  while (i + 1 < m.n && b >= m.first[i + 1]) ++i;
  const int nb = m.first[i + 1] - m.first[i], gx = m.gx[i];
  int h = b - m.first[i];
  if (nb % 8 == 0 && m.first[i] % 8 == 0) h = (h % 8) * (nb / 8) + h / 8;
  wgrad_f32_block<T, E, ROWS, WHOLE>(m.a[i], WgBlock{h % gx, h / gx});
}

// --------------------------------------------------------- bf16 MFMA --
// Weight gradient with bf16 operands on the bf16 MFMA
// (v_mfma_f32_16x16x32_bf16, fp32 accumulate).  The same GEMM as the fp32
// wide layout (rows = 64 output channels, columns = BC input channels x 9
// taps, reduction over the 64 pixels of a tile per LDS stage), but a lane of
// this MFMA supplies 8 consecutive pixels of its row / column, so a tile
// row (TW = 32, 16 or 8 columns) is read in 16-byte pieces:
//   * dy tile in LDS as [k][pixel] (rows of 64 pixels, pitch 72 bf16);
//   * x halo in LDS as [c][halo row][column], stored three times: copy s
//     holds halo columns s .. s+TW-1, i.e. the x values column tap s reads,
//     so the 8 pixels a lane reads at tap (r, s) are 16 aligned bytes of
//     copy s.  Channel planes sit 8 * odd words apart, so the 16 channels of
//     a 16-lane group land in distinct bank groups.
// The four waves split the block's 16-channel column groups (BC / 16 of
// them), its k rows and the two 32-pixel steps of a stage: with BC = 32 a
// wave owns all 64 k x 16 c for one of the two steps, so one B operand read
// from LDS feeds four MFMAs (and an A read nine); with BC = 16, 32 k x 16 c
// for one step.  The two step halves of a wave's columns are summed through
// LDS at the end.  The bias gradient adds the dy operands on the vector ALU
// (bf16 pair dot products against ones, fp32 sums).
//
// Staging moves V consecutive columns per lane (V = 8, 4, 2 when the image
// width is a multiple of V, else 1): one global load of V elements per tile
// row piece, one LDS store per copy.  The copies shifted by one column take
// the missing element from the neighbouring lane (a DPP row shift) or, at
// the tile's left and right edges, from a separate 2-byte load.  A thread
// owns a fixed column piece and a fixed set of rows, so every offset is a
// per-tile base plus a compile-time constant.
template <int TH_, int TW_, int BC_>
struct WgBTile {
  static constexpr int TH = TH_, TW = TW_, BC = BC_;
  static constexpr int BP = TH * TW;                 // pixels per tile
  static_assert(BP == 64 && TW % 8 == 0, "64-pixel tiles of 8-pixel row groups");
  static constexpr int BK = 64;
  static_assert(BC == 16 || BC == 32, "16 or 32 input channels per block");
  static constexpr int WC = BC / 16;                 // waves along c
  static constexpr int WP = 2;                       // waves along the two pixel steps
  static constexpr int WK = 4 / (WC * WP);           // waves along k
  static constexpr int MA = 4 / WK;                  // 16-row blocks of k per wave
  static_assert(WC * WP * WK == 4, "four waves");
  static constexpr int HH = TH + 2;
  static constexpr int PLANE = HH * TW;              // one channel of one copy
  static constexpr int plane_pitch(int p) { return (p / 2) % 8 == 4 ? p : plane_pitch(p + 8); }
  static constexpr int PLANE_P = plane_pitch(PLANE);
  static constexpr int DYP = BP + 8;                 // dy row pitch: 36 words
  static constexpr int LDS_DY = BK * DYP;            // bf16 elements
  static constexpr int LDS_XC = BC * PLANE_P;        // one shifted copy
  static constexpr int LDS_BUF = LDS_DY + 3 * LDS_XC;
  static_assert(PLANE % 8 == 0 && LDS_DY % 8 == 0 && LDS_XC % 8 == 0, "16-byte reads");
  static constexpr size_t LDS_BYTES = 2 * LDS_BUF * sizeof(u16);
  static_assert(LDS_BYTES <= 80 * 1024, "two blocks must fit in the 160 KB of LDS");
};

typedef short s8 __attribute__((ext_vector_type(8)));

// End of a bf16 weight-gradient block (both tile forms): the bias row sums,
// the two pixel-step halves summed (waves wp = 1 hand their accumulators to
// the waves wp = 0 of the same (wk, wc) through LDS), and the block's
// 64 k x (BC c x 9 taps) tile written to dw or to its split's partials.
template <class T>
__device__ __forceinline__ void wgrad_bf16_finish(const WgArgs& a, const WgBlock& blk, int k0,
                                                  int c0, bool do_db, int wk, int wp, int wc,
                                                  f4 (&acc)[T::MA][9], float (&sbias)[T::MA],
                                                  u16* ldsw) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int kq = lane >> 4, lr = lane & 15;
  f4 accb[T::MA];
#pragma unroll
  for (int m = 0; m < T::MA; ++m) accb[m] = wave_row_sums(sbias[m]);

  // Sum the two step halves: waves wp = 1 hand their accumulators to the
  // waves wp = 0 of the same (wk, wc) through LDS (lane fastest, so the
  // stores and loads are conflict-free), in rounds of RA k blocks.
  {
    constexpr int RA =                                 // k blocks per round
        T::MA >= 2 && T::WC * T::WK * 2 * 40 * 64 * 4 <= (int)T::LDS_BYTES ? 2 : 1;
    constexpr int NF = RA * 10 * 4;                    // floats per lane per round
    static_assert(T::WC * T::WK * NF * 64 * 4 <= T::LDS_BYTES, "reduction fits the LDS");
    float* R = reinterpret_cast<float*>(ldsw) + (wk * T::WC + wc) * NF * 64;
#pragma unroll
    for (int r0 = 0; r0 < T::MA; r0 += RA) {
      if (wp == 1) {
#pragma unroll
        for (int m = 0; m < RA; ++m) {
#pragma unroll
          for (int t = 0; t < 9; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) R[((m * 10 + t) * 4 + i) * 64 + lane] = acc[r0 + m][t][i];
#pragma unroll
          for (int i = 0; i < 4; ++i) R[((m * 10 + 9) * 4 + i) * 64 + lane] = accb[r0 + m][i];
        }
      }
      __syncthreads();
      if (wp == 0) {
#pragma unroll
        for (int m = 0; m < RA; ++m) {
#pragma unroll
          for (int t = 0; t < 9; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[r0 + m][t][i] += R[((m * 10 + t) * 4 + i) * 64 + lane];
#pragma unroll
          for (int i = 0; i < 4; ++i) accb[r0 + m][i] += R[((m * 10 + 9) * 4 + i) * 64 + lane];
        }
      }
      __syncthreads();
    }
  }
  // acc[m][t] of the waves wp = 0 holds rows k = k0 + (wk*MA + m)*16 +
  // 4*kq + i and channel c0 + wc*16 + lr.  The block's 64 k x (BC c x 9
  // taps) tile goes out through LDS in rounds of 32 rows of BC * 9
  // consecutive floats (the dw order), written in 16-byte pieces; every
  // wave takes part in the barriers and the stores.
  {
    constexpr int RW = T::BC * 9, RP = RW + 4, ROWS = 32, QPR = RW / 4;
    static_assert(ROWS * RP * sizeof(float) <= T::LDS_BYTES && RW % 4 == 0, "rows fit the LDS");
    float* L = reinterpret_cast<float*>(ldsw);
    const int cw = min(T::BC, a.C - c0) * 9;         // live columns of the tile
    const size_t wsz = (size_t)a.K * a.C * 9;
    float* dst = a.splits == 1 ? a.dw : a.part + (size_t)blk.z * (wsz + a.K);
    const bool vec = (a.C * 9) % 4 == 0 && cw % 4 == 0 &&
                     (((uintptr_t)dst + (size_t)c0 * 9 * sizeof(float)) & 15) == 0;
#pragma unroll
    for (int r0 = 0; r0 < T::BK; r0 += ROWS) {
      __syncthreads();                                // the LDS is free
      if (wp == 0) {
#pragma unroll
        for (int m = 0; m < T::MA; ++m) {
          const int row = (wk * T::MA + m) * 16 - r0;
          if (row < 0 || row >= ROWS) continue;
#pragma unroll
          for (int t = 0; t < 9; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              L[(row + 4 * kq + i) * RP + (wc * 16 + lr) * 9 + t] = acc[m][t][i];
        }
      }
      __syncthreads();
      for (int q = tid; q < ROWS * QPR; q += 256) {
        const int row = q / QPR, col = (q % QPR) * 4, k = k0 + r0 + row;
        if (k >= a.K || col >= cw) continue;
        float* o = dst + (size_t)k * a.C * 9 + (size_t)c0 * 9 + col;
        const float* l = L + row * RP + col;
        if (vec) {
          *reinterpret_cast<f4*>(o) = *reinterpret_cast<const f4*>(l);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (col + e < cw) o[e] = l[e];
        }
      }
    }
    if (wp == 0 && do_db && lr == 0) {
      float* pb = a.splits == 1 ? a.db : dst + wsz;
#pragma unroll
      for (int m = 0; m < T::MA; ++m)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = k0 + (wk * T::MA + m) * 16 + 4 * kq + i;
          if (k < a.K) pb[k] = accb[m][i];
        }
    }
  }
}

template <class T, int V>
__global__ __launch_bounds__(256, 2) void conv3x3_wgrad_bf16(WgArgs a) {
  extern __shared__ u16 ldsw[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kq = lane >> 4, lr = lane & 15;
  const WgBlock blk = wg_block();
  const int ct = blk.x % a.c_tiles, kt = blk.x / a.c_tiles;
  const int c0 = ct * T::BC, k0 = kt * T::BK;
  const int pt0 = blk.z * a.tiles_per_split;
  const int pt1 = min(a.ptiles, pt0 + a.tiles_per_split);
  // wave = (wk, wp, wc), wc fastest.
  const int wc = wave % T::WC, wp = (wave / T::WC) % T::WP, wk = wave / (T::WC * T::WP);
  const bool do_db = (a.db != nullptr) && ct == 0 && wc == 0;
  const int HWs = a.H * a.W;

  f4 acc[T::MA][9];
  float sbias[T::MA];    // this lane's share of the bias gradient of row block m
#pragma unroll
  for (int m = 0; m < T::MA; ++m) {
    sbias[m] = 0.f;
#pragma unroll
    for (int t = 0; t < 9; ++t) acc[m][t] = f4{0.f, 0.f, 0.f, 0.f};
  }

  // Staging geometry: LPR lanes per tile row piece of TW columns, RPI rows
  // per round of 256 threads.  dy rows are (k, tile row), k-major; x rows
  // (halo row, c), c fastest.
  constexpr int VV = V;
  constexpr int LPR = T::TW / VV, RPI = 256 / LPR;
  constexpr int DY_I = T::BK * T::TH / RPI;
  constexpr int XROWS = T::HH * T::BC;
  constexpr int X_I = (XROWS + RPI - 1) / RPI;
  static_assert(RPI % T::TH == 0 && T::BK * T::TH % RPI == 0, "whole dy rounds");
  static_assert(VV == 1 || 16 % LPR == 0, "a tile row piece within one DPP row");
  const int vc = tid % LPR, col = vc * VV, r0 = tid / LPR;
  const int dk = r0 / T::TH, dyy = r0 % T::TH;
  const int kleft = a.K - k0 - dk;

  // Next tile to load, advanced after every load.
  int ntx = pt0 % a.tiles_w, nty = (pt0 / a.tiles_w) % a.tiles_h,
      nn = pt0 / (a.tiles_w * a.tiles_h);

  // Registers holding the tile in flight.
  typedef typename std::conditional<(VV > 1), Vec<(VV > 1 ? VV : 2)>, u16>::type Piece;
  Piece rdy[DY_I], rx[X_I];
  u16 rel[X_I], rer[X_I];

  auto gload = [&]() {
    const int h0 = nty * T::TH, w0 = ntx * T::TW, n0 = nn;
    if (++ntx == a.tiles_w) {
      ntx = 0;
      if (++nty == a.tiles_h) { nty = 0; ++nn; }
    }
    const rsrc_t dr = image_rsrc<u16>(a.dy, n0, 1, a.N, a.K * HWs);
    const rsrc_t xr = image_rsrc<u16>(a.x, n0, 1, a.N, a.C * HWs);
    const bool w_ok = w0 + col < a.W;
    {
      const bool ok = w_ok && h0 + dyy < a.H;
      const int base = (k0 + dk) * HWs + (h0 + dyy) * a.W + w0 + col;
#pragma unroll
      for (int i = 0; i < DY_I; ++i) {
        const int dki = (RPI / T::TH) * i;
        const uint32_t off = ok && dki < kleft ? (uint32_t)(base + dki * HWs) * 2u : kOOB;
        if constexpr (VV > 1) rdy[i] = load_vec<VV>(dr, off);
        else rdy[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(dr, (int)off, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < X_I; ++i) {
      const int r = r0 + RPI * i;
      const int cc = r % T::BC, hy = r / T::BC;
      const int h = h0 - 1 + hy, c = c0 + cc;
      const bool row_ok = (XROWS % RPI == 0 || r < XROWS) && c < a.C &&
                          (unsigned)h < (unsigned)a.H;
      const int rbase = c * HWs + h * a.W + w0;
      // Interior columns col .. col+V-1 of the tile (halo columns col+1 ..).
      const uint32_t off = row_ok && w_ok ? (uint32_t)(rbase + col) * 2u : kOOB;
      if constexpr (VV > 1) rx[i] = load_vec<VV>(xr, off);
      else rx[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(xr, (int)off, 0, 0);
      // Edge columns w0 - 1 (first piece of a row) and w0 + TW (last piece).
      const bool l_ok = row_ok && vc == 0 && w0 > 0;
      const bool r_ok = row_ok && vc == LPR - 1 && w0 + T::TW < a.W;
      if constexpr (LPR == 1) {
        rel[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(
            xr, l_ok ? (int)((uint32_t)(rbase - 1) * 2u) : (int)kOOB, 0, 0);
        rer[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(
            xr, r_ok ? (int)((uint32_t)(rbase + T::TW) * 2u) : (int)kOOB, 0, 0);
      } else {
        const uint32_t eoff = l_ok ? (uint32_t)(rbase - 1) * 2u
                              : r_ok ? (uint32_t)(rbase + T::TW) * 2u : kOOB;
        rel[i] = (u16)__builtin_amdgcn_raw_buffer_load_b16(xr, (int)eoff, 0, 0);
      }
    }
  };
  auto lstore = [&](int buf) {
    u16* Dl = ldsw + buf * T::LDS_BUF;
    u16* Xl = Dl + T::LDS_DY;
    {
      u16* q = Dl + dk * T::DYP + dyy * T::TW + col;
#pragma unroll
      for (int i = 0; i < DY_I; ++i) {
        if constexpr (VV > 1) store_vec<VV>(q + (RPI / T::TH) * i * T::DYP, rdy[i]);
        else q[(RPI / T::TH) * i * T::DYP] = rdy[i];
      }
    }
#pragma unroll
    for (int i = 0; i < X_I; ++i) {
      const int r = r0 + RPI * i;
      if (XROWS % RPI != 0 && r >= XROWS) continue;
      const int cc = r % T::BC, hy = r / T::BC;
      u16* q = Xl + cc * T::PLANE_P + hy * T::TW + col;
      // Copy s at column j holds halo column j + s, i.e. x column
      // w0 + j + s - 1: copy 1 is the loaded piece itself, copy 0 the piece
      // shifted right by one element, copy 2 shifted left by one.
      if constexpr (VV > 1) {
        constexpr int D = VV / 2;
        const Vec<VV>& v = rx[i];
        uint32_t left, right;     // x columns col - 1 and col + V (low 16 bits)
        if constexpr (LPR == 1) {
          left = rel[i];
          right = rer[i];
        } else {
          // 0x111: row_shr:1 (lane - 1), 0x101: row_shl:1 (lane + 1).
          const uint32_t pl = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.d[D - 1], 0x111, 0xf, 0xf, true);
          const uint32_t pr = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.d[0], 0x101, 0xf, 0xf, true);
          left = vc == 0 ? (uint32_t)rel[i] : pl >> 16;
          right = vc == LPR - 1 ? (uint32_t)rel[i] : pr & 0xffffu;
        }
        Vec<VV> s0, s2;
        s0.d[0] = (v.d[0] << 16) | (left & 0xffffu);
#pragma unroll
        for (int j = 1; j < D; ++j) s0.d[j] = (v.d[j] << 16) | (v.d[j - 1] >> 16);
#pragma unroll
        for (int j = 0; j + 1 < D; ++j) s2.d[j] = (v.d[j + 1] << 16) | (v.d[j] >> 16);
        s2.d[D - 1] = (right << 16) | (v.d[D - 1] >> 16);
        store_vec<VV>(q, s0);
        store_vec<VV>(q + T::LDS_XC, v);
        store_vec<VV>(q + 2 * T::LDS_XC, s2);
      } else {
        // One column per lane: copy 0 at col + 1, copy 1 at col, copy 2 at
        // col - 1; the edge columns fill copy 0 at 0 and copy 2 at TW - 1.
        if (col + 1 < T::TW) q[1] = rx[i];
        q[T::LDS_XC] = rx[i];
        if (col >= 1) q[2 * T::LDS_XC - 1] = rx[i];
        if (col == 0) q[0] = rel[i];
        if (col == T::TW - 1) q[2 * T::LDS_XC] = rel[i];
      }
    }
  };
  static_assert(T::BP / 32 == T::WP, "one 32-pixel step per wave and stage");
  auto compute = [&](int buf) {
    const u16* Dl = ldsw + buf * T::LDS_BUF;
    const u16* Xl = Dl + T::LDS_DY;
    {
      // This wave's step wp; lane group kq takes pixels p .. p+7 of it.
      const int p = wp * 32 + 8 * kq;
      const int yy = p / T::TW, xx = p % T::TW;
      s8 av[T::MA];
#pragma unroll
      for (int m = 0; m < T::MA; ++m)
        av[m] = *reinterpret_cast<const s8*>(Dl + ((wk * T::MA + m) * 16 + lr) * T::DYP + p);
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int r = t / 3, sft = t % 3;
        const s8 bv = *reinterpret_cast<const s8*>(Xl + sft * T::LDS_XC +
                                                   (wc * 16 + lr) * T::PLANE_P +
                                                   (yy + r) * T::TW + xx);
#pragma unroll
        for (int m = 0; m < T::MA; ++m)
          acc[m][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, av[m]), __builtin_bit_cast(bf16x8, bv), acc[m][t], 0, 0,
              0);
      }
      // Bias gradient: the 8 dy values of each A operand added into fp32 by
      // four bf16 pair dot products against (1, 1) on the vector ALU.
      typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
      const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int m = 0; m < T::MA; ++m) {
        const bf16x8 v = __builtin_bit_cast(bf16x8, av[m]);
        sbias[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 0, 1), one2,
                                                   sbias[m], false);
        sbias[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 2, 3), one2,
                                                   sbias[m], false);
        sbias[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 4, 5), one2,
                                                   sbias[m], false);
        sbias[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 6, 7), one2,
                                                   sbias[m], false);
      }
    }
  };

  const int nt = pt1 - pt0;
  if (nt > 0) {
    gload();
    lstore(0);
    if (nt > 1) gload();
  }
  __syncthreads();
  for (int t = 0; t < nt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nt) lstore(buf ^ 1);
    if (t + 2 < nt) gload();
    compute(buf);
    __syncthreads();
  }
  wgrad_bf16_finish<T>(a, blk, k0, c0, do_db, wk, wp, wc, acc, sbias, ldsw);
}

// ------------------------------------------------- channel-blocked bf16 --
// Weight gradient of channel-blocked tensors (SB_NCHW8C: 8 consecutive
// channels of a pixel are one 16-byte piece).  The GEMM and the waves' work
// are the NCHW bf16 kernel's (rows 64 k, columns BC channels x 9 taps,
// reduction over 64-pixel tiles, v_mfma_f32_16x16x32_bf16, the two 32-pixel
// steps of a stage on different waves), but the tiles sit in LDS as they sit
// in memory: dy as [pixel][k] and the x halo as [halo pixel][c], staged as
// whole 16-byte pieces (one load and one LDS store each, no transposition,
// no shifted copies: a tap's shift is a whole row of the halo).  A lane of
// this MFMA needs 8 consecutive pixels of one k (or one c); it reads them
// with two LDS transpose loads (ds_read_b64_tr_b16: within each group of 16
// lanes, lane 4a + e receives element e of the 8-byte pieces the lanes
// a, a + 4, a + 8, a + 12 point at), each lane of the group pointing at 4
// consecutive channels of one of 4 consecutive pixels.
template <int TH_, int TW_, int BC_>
struct WgC8Tile {
  static constexpr int TH = TH_, TW = TW_, BC = BC_;
  static constexpr int BP = TH * TW;
  static_assert(BP == 64 && TW % 8 == 0, "64-pixel tiles of 8-pixel row groups");
  static constexpr int BK = 64;
  static_assert(BC == 16 || BC == 32, "16 or 32 input channels per block");
  static constexpr int WC = BC / 16, WP = 2, WK = 4 / (WC * WP), MA = 4 / WK;
  static_assert(WC * WP * WK == 4, "four waves");
  static constexpr int HH = TH + 2, HWD = TW + 2, HPIX = HH * HWD;
  // Row pitches (bf16): a transpose load's 16 lanes read 4 rows x 32 bytes;
  // 144-byte dy rows and (BC + 16) * 2-byte x rows put the 4 rows' bytes on
  // distinct banks.  Both are whole 16-byte pieces.
  static constexpr int DYP = BK + 8, XP = BC + 16;
  static constexpr int LDS_DY = BP * DYP, LDS_X = HPIX * XP;
  static constexpr int LDS_BUF = LDS_DY + LDS_X;
  static constexpr int DY_PIECES = BP * BK / 8, X_PIECES = HPIX * BC / 8;
  static constexpr int DY_I = DY_PIECES / 256, X_I = (X_PIECES + 255) / 256;
  static_assert(DY_PIECES % 256 == 0, "whole rounds of dy pieces");
  // The block's end reuses the LDS for the step-half reduction (up to
  // 2 * 40 floats per lane of each (wk, wc) wave) and the dw row staging
  // (32 rows of BC * 9 + 4 floats).
  static constexpr size_t STAGE = 2 * LDS_BUF * sizeof(u16);
  static constexpr size_t RED = (size_t)WC * WK * 2 * 40 * 64 * 4;
  static constexpr size_t ROWS = (size_t)32 * (BC * 9 + 4) * 4;
  static constexpr size_t LDS_BYTES = STAGE > RED ? (STAGE > ROWS ? STAGE : ROWS)
                                                  : (RED > ROWS ? RED : ROWS);
  static_assert(LDS_BYTES <= 80 * 1024, "two blocks must fit in the 160 KB of LDS");
};

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

// 8 consecutive-row values of one column from two transpose loads: rows
// r0 .. r0 + 3 and r0 + 4 .. r0 + 7 (row pitch `pitch` bf16), the 16-lane
// group's column block at col0 (lane 4a + e of the group gets column
// col0 + 4a + e).  `lrow(j)` maps j = 0..7 to the LDS row.
template <class Row>
__device__ __forceinline__ s8 tr_read8(const u16* base, int pitch, int col0, Row lrow) {
  const int s = threadIdx.x & 15, a = s & 3, j = s >> 2;
  const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4s*)(base + lrow(j) * pitch + col0 + 4 * a));
  const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4s*)(base + lrow(j + 4) * pitch + col0 + 4 * a));
  return s8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// The first half of tr_read8: rows r0 .. r0 + 3 only.
template <class Row>
__device__ __forceinline__ v4s tr_read4(const u16* base, int pitch, int col0, Row lrow) {
  const int s = threadIdx.x & 15, a = s & 3, j = s >> 2;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4s*)(base + lrow(j) * pitch + col0 + 4 * a));
}

template <class T>
__global__ __launch_bounds__(256, 2) void conv3x3_wgrad_c8(WgArgs a) {
  extern __shared__ u16 ldsw[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kq = lane >> 4;
  const WgBlock blk = wg_block();
  const int ct = blk.x % a.c_tiles, kt = blk.x / a.c_tiles;
  const int c0 = ct * T::BC, k0 = kt * T::BK;
  const int pt0 = blk.z * a.tiles_per_split;
  const int pt1 = min(a.ptiles, pt0 + a.tiles_per_split);
  const int wc = wave % T::WC, wp = (wave / T::WC) % T::WP, wk = wave / (T::WC * T::WP);
  const bool do_db = (a.db != nullptr) && ct == 0 && wc == 0;
  const bool do_db_w = __builtin_amdgcn_readfirstlane(do_db ? 1 : 0) != 0;
  const int HWs = a.H * a.W, KB = a.K / 8, CB = a.C / 8;

  f4 acc[T::MA][9];
  float sbias[T::MA];
#pragma unroll
  for (int m = 0; m < T::MA; ++m) {
    sbias[m] = 0.f;
#pragma unroll
    for (int t = 0; t < 9; ++t) acc[m][t] = f4{0.f, 0.f, 0.f, 0.f};
  }

  // Staging: dy piece q = (k block q / 64, tile pixel q % 64); x piece
  // q = (c block q / HPIX, halo pixel q % HPIX).  Offsets (elements) within
  // an image for a tile at (h0, w0) = (0, 0) (negative for the halo's first
  // row or column), and whether the piece's k or c block exists.
  int dy_rel[T::DY_I], dy_yy[T::DY_I], dy_xx[T::DY_I];
  bool dy_live[T::DY_I];
#pragma unroll
  for (int i = 0; i < T::DY_I; ++i) {
    const int q = tid + 256 * i, p = q % 64, kb = k0 / 8 + q / 64;
    dy_yy[i] = p / T::TW;
    dy_xx[i] = p % T::TW;
    dy_live[i] = kb < KB;
    dy_rel[i] = (kb * HWs + dy_yy[i] * a.W + dy_xx[i]) * 8;
  }
  int x_rel[T::X_I], x_hy[T::X_I], x_hx[T::X_I];
  bool x_live[T::X_I];
#pragma unroll
  for (int i = 0; i < T::X_I; ++i) {
    const int q = tid + 256 * i, hp = q % T::HPIX, cb = c0 / 8 + q / T::HPIX;
    x_hy[i] = hp / T::HWD - 1;
    x_hx[i] = hp % T::HWD - 1;
    x_live[i] = q < T::X_PIECES && cb < CB;
    x_rel[i] = (cb * HWs + x_hy[i] * a.W + x_hx[i]) * 8;
  }

  int ntx = pt0 % a.tiles_w, nty = (pt0 / a.tiles_w) % a.tiles_h,
      nn = pt0 / (a.tiles_w * a.tiles_h);
  s8 rdy[T::DY_I], rx[T::X_I];

  auto gload = [&]() {
    const int h0 = nty * T::TH, w0 = ntx * T::TW, n0 = nn;
    if (++ntx == a.tiles_w) {
      ntx = 0;
      if (++nty == a.tiles_h) { nty = 0; ++nn; }
    }
    const rsrc_t dr = image_rsrc<u16>(a.dy, n0, 1, a.N, a.K * HWs);
    const rsrc_t xr = image_rsrc<u16>(a.x, n0, 1, a.N, a.C * HWs);
    const int tile = (h0 * a.W + w0) * 8;
#pragma unroll
    for (int i = 0; i < T::DY_I; ++i) {
      const bool ok = dy_live[i] && h0 + dy_yy[i] < a.H && w0 + dy_xx[i] < a.W;
      const uint32_t off = ok ? (uint32_t)(dy_rel[i] + tile) * 2u : kOOB;
      rdy[i] = __builtin_bit_cast(s8, __builtin_amdgcn_raw_buffer_load_b128(dr, (int)off, 0, 0));
    }
#pragma unroll
    for (int i = 0; i < T::X_I; ++i) {
      const bool ok = x_live[i] && (unsigned)(h0 + x_hy[i]) < (unsigned)a.H &&
                      (unsigned)(w0 + x_hx[i]) < (unsigned)a.W;
      const uint32_t off = ok ? (uint32_t)(x_rel[i] + tile) * 2u : kOOB;
      rx[i] = __builtin_bit_cast(s8, __builtin_amdgcn_raw_buffer_load_b128(xr, (int)off, 0, 0));
    }
  };
  auto lstore = [&](int buf) {
    u16* Dl = ldsw + buf * T::LDS_BUF;
    u16* Xl = Dl + T::LDS_DY;
#pragma unroll
    for (int i = 0; i < T::DY_I; ++i) {
      const int q = tid + 256 * i;
      *reinterpret_cast<s8*>(Dl + (q % 64) * T::DYP + (q / 64) * 8) = rdy[i];
    }
#pragma unroll
    for (int i = 0; i < T::X_I; ++i) {
      const int q = tid + 256 * i;
      if (q < T::X_PIECES)
        *reinterpret_cast<s8*>(Xl + (q % T::HPIX) * T::XP + (q / T::HPIX) * 8) = rx[i];
    }
  };
  auto compute = [&](int buf) {
    const u16* Dl = ldsw + buf * T::LDS_BUF;
    const u16* Xl = Dl + T::LDS_DY;
    // This wave's step wp; lane group kq takes pixels p .. p + 7 (one row).
    const int p = wp * 32 + 8 * kq;
    const int yy = p / T::TW, xx = p % T::TW;
    s8 av[T::MA];
#pragma unroll
    for (int m = 0; m < T::MA; ++m)
      av[m] = tr_read8(Dl, T::DYP, (wk * T::MA + m) * 16, [&](int j) { return p + j; });
    // The three taps of a filter row read the same halo row at column
    // offsets 0, 1, 2: the lane's 8 pixels at offset 0 are read once, with
    // the next 4 (of which the first 2 are used; a lane whose columns would
    // pass the row's end reads its last column instead), and the windows at
    // offsets 1 and 2 are shifted out of those 12 values in registers.
    s8 rb[3];
    v4s rn[3];
    auto rrow = [&](int r) {
      rb[r] = tr_read8(Xl, T::XP, wc * 16, [&](int j) { return (yy + r) * T::HWD + xx + j; });
      rn[r] = tr_read4(Xl, T::XP, wc * 16, [&](int j) {
        return (yy + r) * T::HWD + min(xx + 8 + j, T::HWD - 1);
      });
    };
    rrow(0);
#pragma unroll
    for (int r = 0; r < 3; ++r) {
      if (r + 1 < 3) rrow(r + 1);
      __builtin_amdgcn_sched_barrier(0);
      const s8 b0 = rb[r];
      const v4s nx = rn[r];
      const s8 b1 = s8{b0[1], b0[2], b0[3], b0[4], b0[5], b0[6], b0[7], nx[0]};
      const s8 b2 = s8{b0[2], b0[3], b0[4], b0[5], b0[6], b0[7], nx[0], nx[1]};
#pragma unroll
      for (int sft = 0; sft < 3; ++sft) {
        const s8 bv = sft == 0 ? b0 : sft == 1 ? b1 : b2;
#pragma unroll
        for (int m = 0; m < T::MA; ++m)
          acc[m][r * 3 + sft] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, av[m]), __builtin_bit_cast(bf16x8, bv),
              acc[m][r * 3 + sft], 0, 0, 0);
      }
    }
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
    // Only the waves that write db sum it (the same for a whole wave).
    if (do_db_w)
#pragma unroll
    for (int m = 0; m < T::MA; ++m) {
      const bf16x8 v = __builtin_bit_cast(bf16x8, av[m]);
      sbias[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 0, 1), one2,
                                                 sbias[m], false);
      sbias[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 2, 3), one2,
                                                 sbias[m], false);
      sbias[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 4, 5), one2,
                                                 sbias[m], false);
      sbias[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 6, 7), one2,
                                                 sbias[m], false);
    }
  };

  const int nt = pt1 - pt0;
  if (nt > 0) {
    gload();
    lstore(0);
    if (nt > 1) gload();
  }
  __syncthreads();
  for (int t = 0; t < nt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nt) lstore(buf ^ 1);
    if (t + 2 < nt) gload();
    compute(buf);
    __syncthreads();
  }
  wgrad_bf16_finish<T>(a, blk, k0, c0, do_db, wk, wp, wc, acc, sbias, ldsw);
}

// ------------------------------------------------------ small whole images --
template <int H_, int W_, int IW_>
struct WgSmall {
  static constexpr int H = H_, W = W_, P = H * W, IW = IW_;   // IW images per LDS fill
  static constexpr int BK = 64, BC = 16;
  static constexpr int DZ_STRIDE = BK + 16;                    // per (position, image)
  static constexpr int LDS_DZ = P * IW * DZ_STRIDE;
  static constexpr int LDS_X = P * IW * BC;
  static constexpr int LDS_BUF = LDS_DZ + LDS_X;
  static constexpr size_t LDS_BYTES = 2 * LDS_BUF * sizeof(float);
  static_assert(P % 4 == 0 && IW % 4 == 0, "float4 planes, 4-image MFMA steps");
  static constexpr int DZ_F4 = IW * BK * P / 4;
  static constexpr int X_F4 = IW * BC * P / 4;
  static constexpr int DZ_PT = DZ_F4 / 256;
  static constexpr int X_PT = X_F4 / 256;
  // Every staging lane is live: the stores need no condition.
  static_assert(DZ_F4 % 256 == 0 && X_F4 % 256 == 0, "staging covers whole 256-thread rounds");
  __host__ __device__ static constexpr int src(int pos, int tap) {
    return (pos / W + tap / 3 - 1 >= 0 && pos / W + tap / 3 - 1 < H &&
            pos % W + tap % 3 - 1 >= 0 && pos % W + tap % 3 - 1 < W)
               ? (pos / W + tap / 3 - 1) * W + (pos % W + tap % 3 - 1)
               : -1;
  }
};

template <class T, class E>
__global__ __launch_bounds__(256, 2) void conv3x3_wgrad_small_f32(WgArgs a) {
  extern __shared__ float lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int jq = lane >> 4, lr = lane & 15;
  const WgBlock blk = wg_block();
  const int ct = blk.x % a.c_tiles, kt = blk.x / a.c_tiles;
  const int c0 = ct * T::BC, k0 = kt * T::BK;
  const int ch0 = blk.z * a.tiles_per_split;              // image chunks of IW
  const int ch1 = min(a.ptiles, ch0 + a.tiles_per_split);
  const bool do_db = (a.db != nullptr) && ct == 0;

  // float4 q of a chunk = (image, channel, quarter); quarter fastest.
  int dz_off[T::DZ_PT], dz_loff[T::DZ_PT];
#pragma unroll
  for (int i = 0; i < T::DZ_PT; ++i) {
    int q = tid + i * 256;
    int kk = q % T::BK, rest = q / T::BK;          // k fastest: conflict-free LDS rows
    int quarter = rest % (T::P / 4), img = rest / (T::P / 4);
    bool ok = k0 + kk < a.K;
    dz_off[i] = ok ? (img * a.K + k0 + kk) * T::P + quarter * 4 : -1;   // from the chunk's first image
    dz_loff[i] = ((quarter * 4) * T::IW + img) * T::DZ_STRIDE + kk;
  }
  int x_off[T::X_PT], x_loff[T::X_PT];
#pragma unroll
  for (int i = 0; i < T::X_PT; ++i) {
    int q = tid + i * 256;
    int cc = q % T::BC, rest = q / T::BC;          // c, then image: consecutive LDS rows
    int img = rest % T::IW, quarter = rest / T::IW;
    bool ok = c0 + cc < a.C;
    x_off[i] = ok ? (img * a.C + c0 + cc) * T::P + quarter * 4 : -1;    // from the chunk's first image
    x_loff[i] = ((quarter * 4) * T::IW + img) * T::BC + cc;
  }

  f4 acc[9];
  float sbias = 0.f;     // this lane's share of its row's bias gradient
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};

  f4 rdz[T::DZ_PT], rx[T::X_PT];
  auto gload = [&](int ch) {
    const int nb = ch * T::IW;                        // first image of the chunk
    const rsrc_t dr = image_rsrc<E>(a.dy, nb, T::IW, a.N, a.K * T::P);
    const rsrc_t xr = image_rsrc<E>(a.x, nb, T::IW, a.N, a.C * T::P);
#pragma unroll
    for (int i = 0; i < T::DZ_PT; ++i) {
      const int img = (tid + i * 256) / T::BK / (T::P / 4);
      const bool ok = dz_off[i] >= 0 && nb + img < a.N;
      rdz[i] = BufLoad<E>::four(dr, ok ? (uint32_t)dz_off[i] * (uint32_t)sizeof(E) : kOOB);
    }
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) {
      const int img = (tid + i * 256) / T::BC % T::IW;
      const bool ok = x_off[i] >= 0 && nb + img < a.N;
      rx[i] = BufLoad<E>::four(xr, ok ? (uint32_t)x_off[i] * (uint32_t)sizeof(E) : kOOB);
    }
  };
  auto lstore = [&](int buf) {
    float* Dl = lds + buf * T::LDS_BUF;
    float* Xl = Dl + T::LDS_DZ;
#pragma unroll
    for (int i = 0; i < T::DZ_PT; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) Dl[dz_loff[i] + j * T::IW * T::DZ_STRIDE] = rdz[i][j];
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) Xl[x_loff[i] + j * T::IW * T::BC] = rx[i][j];
  };
  auto compute = [&](int buf) {
    const float* Dl = lds + buf * T::LDS_BUF;
    const float* Xl = Dl + T::LDS_DZ;
#pragma unroll
    for (int s = 0; s < T::IW / 4; ++s) {
      float av[T::P], bv[T::P];
#pragma unroll
      for (int pos = 0; pos < T::P; ++pos) {
        av[pos] = Dl[(pos * T::IW + 4 * s + jq) * T::DZ_STRIDE + wave * 16 + lr];
        bv[pos] = Xl[(pos * T::IW + 4 * s + jq) * T::BC + lr];
      }
#pragma unroll
      for (int pos = 0; pos < T::P; ++pos) {
#pragma unroll
        for (int t = 0; t < 9; ++t) {
          const int sp = T::src(pos, t);
          if (sp >= 0) acc[t] = mfma16x16x4(av[pos], bv[sp], acc[t]);
        }
        sbias += av[pos];
      }
    }
  };

  const int nt = ch1 - ch0;
  if (nt > 0) {
    gload(ch0);
    lstore(0);
    if (nt > 1) gload(ch0 + 1);
  }
  __syncthreads();
  for (int t = 0; t < nt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nt) lstore(buf ^ 1);
    if (t + 2 < nt) gload(ch0 + t + 2);
    compute(buf);
    __syncthreads();
  }

  static_assert(64 * (16 * 9 + 4) * sizeof(float) <= T::LDS_BYTES, "tile fits the LDS");
  wgrad_store_rows(a, blk.z, k0, c0, do_db, wave_row_sums(sbias), acc, lds);
}

// ------------------------------------------------- 2x2 images: one GEMM --
// At 2x2 every input position lies in the 3x3 window of every output
// position, so all 16 (output position p, input position q) pairs of an
// image are taps inside the image, and the weight gradient is a dense
// product over the images,
//   G[(k,p)][(c,q)] = sum_n dy[n][k][p] * x[n][c][q],
// whose rows (k,p) and columns (c,q) follow dy's and x's NCHW order, folded
// afterwards: dW[k][c][r][s] sums G over the pairs with q = p + (r-1, s-1).
// No MFMA is spent on padding.  Block tile 128 rows (32 k) x 128 columns
// (32 c), four waves of 64 x 64 (4 x 4 blocks of the 16x16x4 MFMA), 32
// images per LDS stage, double-buffered; both operands are staged as
// [image][row] with 16-byte loads of 4 consecutive rows.  The fold runs in
// the epilogue through LDS (G is never written out); the bias gradient is
// summed from the dy operands on the vector ALU and written by the first
// column tile's blocks.  Splits over the images write partials as the other
// weight-gradient kernels do.
struct Wg2 {
  static constexpr int BM = 128, BN = 128, BI = 32;
  static constexpr int RS = BM + 4;                 // [image][row] stride: 4*RS = 16 mod 64 banks
  static constexpr int OP = BI * RS;                // floats per operand stage
  static constexpr int KS = 260;                    // fold tile: [k 16][c 16][p 4][q 4], k stride
  static constexpr int FOLD = 16 * KS;              // floats per wave
  static constexpr int LDS_FLOATS = 4 * OP > 4 * FOLD ? 4 * OP : 4 * FOLD;
  static constexpr size_t LDS_BYTES = LDS_FLOATS * sizeof(float);
};

template <class E>
__global__ __launch_bounds__(256, 2) void conv3x3_wgrad_2x2(WgArgs a) {
  using T = Wg2;
  extern __shared__ float lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int kq = lane >> 4, lr = lane & 15;
  const WgBlock blk = wg_block();
  const int ct = blk.x % a.c_tiles, kt = blk.x / a.c_tiles;
  const int M = a.K * 4, NC = a.C * 4;              // rows and columns of G
  const int m0 = kt * T::BM, n0 = ct * T::BN;
  const int s0 = blk.z * a.tiles_per_split;         // image stages of BI
  const int s1 = min(a.ptiles, s0 + a.tiles_per_split);
  const bool do_db = a.db != nullptr && ct == 0 && wn == 0;   // wave-uniform

  f4 acc[4][4];
  float sbias[4];        // this lane's share of the bias gradient of rows i*16 + lr
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sbias[i] = 0.f;
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[i][n] = f4{0.f, 0.f, 0.f, 0.f};
  }

  // Staging group g = tid + 256 i: image g / 32, rows 4 (g % 32) .. +3.
  f4 ra[4], rb[4];
  auto gload = [&](int s) {
    const int nb = s * T::BI;
    const rsrc_t dr = image_rsrc<E>(a.dy, nb, T::BI, a.N, M);
    const rsrc_t xr = image_rsrc<E>(a.x, nb, T::BI, a.N, NC);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = tid + i * 256, img = g >> 5, r4 = (g & 31) * 4;
      const bool iok = nb + img < a.N;
      ra[i] = BufLoad<E>::four(
          dr, iok && m0 + r4 < M ? (uint32_t)(img * M + m0 + r4) * (uint32_t)sizeof(E) : kOOB);
      rb[i] = BufLoad<E>::four(
          xr, iok && n0 + r4 < NC ? (uint32_t)(img * NC + n0 + r4) * (uint32_t)sizeof(E) : kOOB);
    }
  };
  auto lstore = [&](int buf) {
    float* A = lds + buf * 2 * T::OP;
    float* B = A + T::OP;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = tid + i * 256, off = (g >> 5) * T::RS + (g & 31) * 4;
      *reinterpret_cast<f4*>(A + off) = ra[i];
      *reinterpret_cast<f4*>(B + off) = rb[i];
    }
  };
  // MFMA k-step j of a 16-image slice takes image 16 s + 4 kq + j from lane
  // group kq, for both operands.
  auto compute = [&](int buf) {
    const float* A = lds + buf * 2 * T::OP;
    const float* B = A + T::OP;
#pragma unroll
    for (int s = 0; s < T::BI / 16; ++s) {
      float fa[4][4], fb[4][4];
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = (s * 16 + kq * 4 + j) * T::RS + b * 16 + lr;
          fa[b][j] = A[r + wm * 64];
          fb[b][j] = B[r + wn * 64];
        }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int n = 0; n < 4; ++n) acc[i][n] = mfma16x16x4(fa[i][j], fb[n][j], acc[i][n]);
#pragma unroll
        for (int i = 0; i < 4; ++i) sbias[i] += fa[i][j];
      }
    }
  };

  const int nt = s1 - s0;
  if (nt > 0) {
    gload(s0);
    lstore(0);
    if (nt > 1) gload(s0 + 1);
  }
  __syncthreads();
  for (int t = 0; t < nt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nt) lstore(buf ^ 1);
    if (t + 2 < nt) gload(s0 + t + 2);
    compute(buf);
    __syncthreads();
  }

  // acc[i][n] element e is G at row wm*64 + i*16 + 4*kq + e of the block
  // (k = 4i + kq of the wave's 16, p = e) and column wn*64 + n*16 + lr
  // (c = 4n + lr/4 of the wave's 16, q = lr % 4): the wave's fold tile.
  float* F = lds + wave * T::FOLD;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int n = 0; n < 4; ++n)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        F[(i * 4 + kq) * T::KS + (n * 4 + (lr >> 2)) * 16 + e * 4 + (lr & 3)] = acc[i][n][e];
  __syncthreads();
  const size_t wsz = (size_t)a.K * a.C * 9;
  float* out = a.splits == 1 ? a.dw : a.part + (size_t)blk.z * (wsz + a.K);
  const int kb = (m0 >> 2) + wm * 16, cb = (n0 >> 2) + wn * 16;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int pr = lane + 64 * r, kl = pr >> 4, cl = pr & 15;
    const float* g = F + kl * T::KS + cl * 16;
    float t9[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) t9[t] = 0.f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const f4 gp = *reinterpret_cast<const f4*>(g + p * 4);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        t9[((q >> 1) - (p >> 1) + 1) * 3 + ((q & 1) - (p & 1) + 1)] += gp[q];
    }
    const int k = kb + kl, c = cb + cl;
    if (k < a.K && c < a.C) {
#pragma unroll
      for (int t = 0; t < 9; ++t) out[((size_t)k * a.C + c) * 9 + t] = t9[t];
    }
  }
  // Bias gradient: row i*16 + lr of the wave is (k = 4i + lr/4, p = lr%4);
  // sum over the lane groups (images), then over p (a fixed butterfly).
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v = sbias[i];
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 32, 64);
    v += __shfl_xor(v, 1, 64);
    v += __shfl_xor(v, 2, 64);
    const int k = kb + i * 4 + (lr >> 2);
    if (do_db && kq == 0 && (lr & 3) == 0 && k < a.K) {
      if (a.splits == 1) a.db[k] = v;
      else out[wsz + k] = v;
    }
  }
}

// ---------------------------------------------------------------- host --
struct WgPlan {
  int imgs;          // images per pixel tile (per LDS fill for the small kernels)
  int tile, tiles_w, tiles_h, ptiles, k_tiles, c_tiles, tps, splits;
  int bc;            // input channels per block of the bf16 MFMA kernel, 0 if not taken
  size_t ws_bytes;
};

using WgW32 = WgTile<2, 32, 1, 0>;
using WgW16 = WgTile<4, 16, 1, 0>;
using WgW8 = WgTile<8, 8, 1, 0>;
using WgW4 = WgTile<4, 4, 4, 0>;
using WgW2 = WgTile<2, 2, 16, 0>;
using WgN32_2 = WgTile<2, 32, 1, 2>;   // C <= 3
using WgN32_4 = WgTile<2, 32, 1, 4>;   // C <= 7
using WgN4_2 = WgTile<4, 4, 4, 2>;
using WgN4_4 = WgTile<4, 4, 4, 4>;
using WgS4 = WgSmall<4, 4, 4>;

static const char* kWgNames[] = {
    "sb::conv3x3_wgrad_f32<sb::WgTile<2, 32, 1, 0>, %s>", "sb::conv3x3_wgrad_f32<sb::WgTile<4, 16, 1, 0>, %s>",
    "sb::conv3x3_wgrad_f32<sb::WgTile<8, 8, 1, 0>, %s>",  "sb::conv3x3_wgrad_f32<sb::WgTile<4, 4, 4, 0>, %s>",
    "sb::conv3x3_wgrad_f32<sb::WgTile<2, 2, 16, 0>, %s>", "sb::conv3x3_wgrad_f32<sb::WgTile<2, 32, 1, 2>, %s>",
    "sb::conv3x3_wgrad_f32<sb::WgTile<2, 32, 1, 4>, %s>", "sb::conv3x3_wgrad_f32<sb::WgTile<4, 4, 4, 2>, %s>",
    "sb::conv3x3_wgrad_f32<sb::WgTile<4, 4, 4, 4>, %s>",
    "sb::conv3x3_wgrad_2x2<%s>",
    "sb::conv3x3_wgrad_small_f32<sb::WgSmall<4, 4, 4>, %s>",
};

// allow_small: the whole-image kernel needs tensors aligned for 4-element moves.
// bf16: the wide tiles (0..2) run on the bf16 MFMA kernel.
static WgPlan wg_plan(int N, int C, int H, int W, int K, bool allow_small, bool bf16) {
  WgPlan p{};
  int th = 2, tw = 32, imgs = 1;
  // bf16 images at least 8 wide take the bf16 MFMA kernel whatever C.
  const bool narrow = C <= 7 && !(bf16 && W >= 8);
  if (narrow) {
    // 32-wide rows for wide images, 4x4 x 4-image tiles otherwise.
    if (W >= 32) { p.tile = C <= 3 ? 5 : 6; }
    else { th = 4; tw = 4; imgs = 4; p.tile = C <= 3 ? 7 : 8; }
  } else if (allow_small && H == 2 && W == 2) { p.tile = 9; th = 2; tw = 2; imgs = Wg2::BI; }
  else if (allow_small && H == 4 && W == 4) { p.tile = 10; th = 4; tw = 4; imgs = 4; }
  else if (W >= 32) { p.tile = 0; }
  else if (W >= 16) { p.tile = 1; th = 4; tw = 16; }
  else if (W >= 8) { p.tile = 2; th = 8; tw = 8; }
  else if (W >= 4) { p.tile = 3; th = 4; tw = 4; imgs = 4; }
  else { p.tile = 4; th = 2; tw = 2; imgs = 16; }
  p.imgs = imgs;
  p.tiles_w = cdiv(W, tw);
  p.tiles_h = cdiv(H, th);
  p.ptiles = p.tiles_w * p.tiles_h * cdiv(N, imgs);   // for the small kernels: image chunks
  p.k_tiles = cdiv(K, 64);
  p.bc = bf16 && p.tile <= 2 ? (C >= 32 ? 32 : 16) : 0;
  p.c_tiles = narrow ? 1 : cdiv(C, p.bc ? p.bc : 16);
  if (p.tile == 9) {                      // 32 k x 32 c per block
    p.k_tiles = cdiv(K, 32);
    p.c_tiles = cdiv(C, 32);
  }
  long blocks = (long)p.k_tiles * p.c_tiles;
  // About two blocks per CU (one for the 2x2 GEMM, whose splits would each
  // write a whole dW), at most 512 splits of the pixel range (a layer of
  // one block, the first layer, then still fills every CU twice).
  const long target = p.tile == 9 ? 256 : 512;
  int splits = 1;
  if (blocks < target)
    splits = (int)std::min<long>(std::min<long>(p.ptiles, 512), cdiv((int)target, (int)blocks));
  p.tps = cdiv(p.ptiles, splits);
  p.splits = cdiv(p.ptiles, p.tps);
  p.ws_bytes = p.splits > 1 ? (size_t)p.splits * ((size_t)K * C * 9 + K) * sizeof(float) : 0;
  return p;
}

template <class E>
static void wg_launch_2x2(const WgPlan& p, const WgArgs& a, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)conv3x3_wgrad_2x2<E>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)Wg2::LDS_BYTES);
    attr_set = true;
  }
  dim3 grid(p.k_tiles * p.c_tiles, 1, p.splits);
  conv3x3_wgrad_2x2<E><<<grid, 256, Wg2::LDS_BYTES, st>>>(a);
  if (p.splits > 1) launch_splits_reduce(a.part, p.splits, a.K, a.C, a.dw, a.db, st);
}

template <class T, bool SMALL, class E, bool ROWS = false, bool WHOLE = false>
static void wg_launch(const WgPlan& p, const WgArgs& a, hipStream_t st) {
  static bool attr_set = false;
  const void* fn;
  if constexpr (SMALL) fn = (const void*)conv3x3_wgrad_small_f32<T, E>;
  else fn = (const void*)conv3x3_wgrad_f32<T, E, ROWS, WHOLE>;
  if (!attr_set) {
    (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
    attr_set = true;
  }
  dim3 grid(p.k_tiles * p.c_tiles, 1, p.splits);
  if constexpr (SMALL)
    conv3x3_wgrad_small_f32<T, E><<<grid, 256, T::LDS_BYTES, st>>>(a);
  else
    conv3x3_wgrad_f32<T, E, ROWS, WHOLE><<<grid, 256, T::LDS_BYTES, st>>>(a);
  if (p.splits > 1) launch_splits_reduce(a.part, p.splits, a.K, a.C, a.dw, a.db, st);
}

// n (<= kWgMany) layers' weight gradients on one launch of
// conv3x3_wgrad_f32_many, then each layer's split reduction in layer order.
template <class T, class E, bool ROWS, bool WHOLE>
static void wg_launch_many(const WgPlan* p, const WgArgs* a, int n, hipStream_t st) {
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute((const void*)conv3x3_wgrad_f32_many<T, E, ROWS, WHOLE>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
  });
  WgMany m{};
  m.n = n;
  int total = 0;
  for (int i = 0; i < n; ++i) {
    m.a[i] = a[i];
    m.first[i] = total;
    m.gx[i] = p[i].k_tiles * p[i].c_tiles;
    total += m.gx[i] * p[i].splits;
  }
  for (int i = n; i <= kWgMany; ++i) m.first[i] = total;
  conv3x3_wgrad_f32_many<T, E, ROWS, WHOLE><<<total, 256, T::LDS_BYTES, st>>>(m);
  for (int i = 0; i < n; ++i)
    if (p[i].splits > 1)
      launch_splits_reduce(a[i].part, p[i].splits, a[i].K, a[i].C, a[i].dw, a[i].db, st);
}

}  // namespace sb

namespace sbh {

// Columns per staging load of the bf16 kernel: the largest of 8, 4, 2 that
// divides the image width and the tile width and keeps both tensors' loads
// aligned, else 1.
static int wg_bf16_vec(int W, const void* x, const void* dy) {
  const uintptr_t u = (uintptr_t)x | (uintptr_t)dy;
  for (int v = 8; v >= 2; v /= 2)
    if (W % v == 0 && (u % (2 * v)) == 0) return v;
  return 1;
}

size_t conv_wgrad_ws(int dtype, int N, int C, int H, int W, int K) {
  const bool bf16 = dtype == SB_BF16;
  return std::max(sb::wg_plan(N, C, H, W, K, true, bf16).ws_bytes,
                  sb::wg_plan(N, C, H, W, K, false, bf16).ws_bytes);
}

int conv_wgrad_describe(int dtype, int N, int C, int H, int W, int K, char* buf, size_t len) {
  sb::WgPlan p = sb::wg_plan(N, C, H, W, K, true, dtype == SB_BF16);
  char name[160];
  static const char* kBTiles[] = {"2, 32", "4, 16", "8, 8"};
  // The bf16 kernel's staging width as for aligned tensors.
  if (p.bc)
    snprintf(name, sizeof(name), "sb::conv3x3_wgrad_bf16<sb::WgBTile<%s, %d>, %d>",
             kBTiles[p.tile], p.bc, wg_bf16_vec(W, nullptr, nullptr));
  else
    snprintf(name, sizeof(name), sb::kWgNames[p.tile],
             dtype == SB_BF16 ? "unsigned short" : "float");
  return snprintf(buf, len, "%s grid=%dx1x%d", name, p.k_tiles * p.c_tiles, p.splits);
}

// The bf16 weight gradient on the bf16 MFMA, for the wide 64-pixel tiles;
// V columns per staging load.
template <class T, int V>
static void wg_launch_bf16(const sb::WgPlan& p, const sb::WgArgs& a, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)sb::conv3x3_wgrad_bf16<T, V>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
    attr_set = true;
  }
  dim3 grid(p.k_tiles * p.c_tiles, 1, p.splits);
  sb::conv3x3_wgrad_bf16<T, V><<<grid, 256, T::LDS_BYTES, st>>>(a);
  if (p.splits > 1) sb::launch_splits_reduce(a.part, p.splits, a.K, a.C, a.dw, a.db, st);
}

template <class T>
static void wg_launch_bf16v(int v, const sb::WgPlan& p, const sb::WgArgs& a, hipStream_t st) {
  switch (v) {
    case 8: wg_launch_bf16<T, 8>(p, a, st); break;
    case 4: wg_launch_bf16<T, 4>(p, a, st); break;
    case 2: wg_launch_bf16<T, 2>(p, a, st); break;
    default: wg_launch_bf16<T, 1>(p, a, st); break;
  }
}

template <class E>
static void wg_dispatch(const sb::WgPlan& p, const sb::WgArgs& a, hipStream_t st) {
  switch (p.tile) {
    // Images exactly as wide as the tile take the full-width staging.
    case 0:
      if (a.W == 32) sb::wg_launch<sb::WgW32, false, E, true>(p, a, st);
      else sb::wg_launch<sb::WgW32, false, E>(p, a, st);
      break;
    case 1:
      if (a.W == 16) sb::wg_launch<sb::WgW16, false, E, true>(p, a, st);
      else sb::wg_launch<sb::WgW16, false, E>(p, a, st);
      break;
    case 2:
      if (a.W == 8 && a.H == 8) sb::wg_launch<sb::WgW8, false, E, true, true>(p, a, st);
      else if (a.W == 8) sb::wg_launch<sb::WgW8, false, E, true>(p, a, st);
      else sb::wg_launch<sb::WgW8, false, E>(p, a, st);
      break;
    case 3: sb::wg_launch<sb::WgW4, false, E>(p, a, st); break;
    case 4: sb::wg_launch<sb::WgW2, false, E>(p, a, st); break;
    case 5: sb::wg_launch<sb::WgN32_2, false, E>(p, a, st); break;
    case 6: sb::wg_launch<sb::WgN32_4, false, E>(p, a, st); break;
    case 7: sb::wg_launch<sb::WgN4_2, false, E>(p, a, st); break;
    case 8: sb::wg_launch<sb::WgN4_4, false, E>(p, a, st); break;
    case 9: sb::wg_launch_2x2<E>(p, a, st); break;
    default: sb::wg_launch<sb::WgS4, true, E>(p, a, st); break;
  }
}

sb_status conv_wgrad(int dtype, int N, int C, int H, int W, int K, const void* x, const void* dy,
                     float* dw, float* db, void* ws, size_t ws_bytes, hipStream_t st) {
  // The whole-image kernel moves 4 elements at a time (16 bytes in fp32, 8
  // in bf16).
  const uintptr_t amask = dtype == SB_BF16 ? 7 : 15;
  const bool aligned = (((uintptr_t)x | (uintptr_t)dy) & amask) == 0;
  sb::WgPlan p = sb::wg_plan(N, C, H, W, K, aligned, dtype == SB_BF16);
  // Buffer ranges: one tile's images of x and of dy.
  if ((int64_t)std::min(p.imgs, N) * std::max(C, K) * H * W * dsize(dtype) >= (1ll << 31))
    return SB_ERR_UNSUPPORTED;
  if (p.ws_bytes > 0 && (ws == nullptr || ws_bytes < p.ws_bytes)) return SB_ERR_WORKSPACE;
  sb::WgArgs a{};
  a.x = x; a.dy = dy; a.dw = dw; a.db = db;
  a.part = p.splits > 1 ? (float*)ws : nullptr;
  a.N = N; a.C = C; a.H = H; a.W = W; a.K = K;
  a.tiles_w = p.tiles_w; a.tiles_h = p.tiles_h; a.ptiles = p.ptiles;
  a.tiles_per_split = p.tps; a.c_tiles = p.c_tiles; a.splits = p.splits;
  const int v = p.bc ? wg_bf16_vec(W, x, dy) : 1;
  if (p.bc == 32) {
    switch (p.tile) {
      case 0: wg_launch_bf16v<sb::WgBTile<2, 32, 32>>(v, p, a, st); break;
      case 1: wg_launch_bf16v<sb::WgBTile<4, 16, 32>>(v, p, a, st); break;
      default: wg_launch_bf16v<sb::WgBTile<8, 8, 32>>(v, p, a, st); break;
    }
  } else if (p.bc == 16) {
    switch (p.tile) {
      case 0: wg_launch_bf16v<sb::WgBTile<2, 32, 16>>(v, p, a, st); break;
      case 1: wg_launch_bf16v<sb::WgBTile<4, 16, 16>>(v, p, a, st); break;
      default: wg_launch_bf16v<sb::WgBTile<8, 8, 16>>(v, p, a, st); break;
    }
  } else if (dtype == SB_BF16) {
    wg_dispatch<sb::u16>(p, a, st);
  } else {
    wg_dispatch<float>(p, a, st);
  }
  return launch_status();
}

// Batch key of an NCHW weight gradient: layers whose plan runs the same
// conv3x3_wgrad_f32 instantiation (fp32, wide tiles) share a key; -1 for a
// layer that takes another kernel (it runs on its own).
int conv_wgrad_batch_key(int dtype, int N, int C, int H, int W, int K, const void* x,
                         const void* dy) {
  if (dtype != SB_F32) return -1;
  const bool aligned = (((uintptr_t)x | (uintptr_t)dy) & 15) == 0;
  const sb::WgPlan p = sb::wg_plan(N, C, H, W, K, aligned, false);
  if (p.bc != 0 || p.tile > 2) return -1;
  if ((int64_t)std::min(p.imgs, N) * std::max(C, K) * H * W * 4 >= (1ll << 31)) return -1;
  const bool rows = (p.tile == 0 && W == 32) || (p.tile == 1 && W == 16) ||
                    (p.tile == 2 && W == 8);
  const bool whole = p.tile == 2 && W == 8 && H == 8;
  return p.tile * 4 + (rows ? 2 : 0) + (whole ? 1 : 0);
}

// n (1..4) layers with one batch key on one launch: the same partials,
// reductions and results as n conv_wgrad calls.  shape[i] = {N, C, H, W, K};
// ws[i] / ws_bytes[i]: layer i's own workspace region.
sb_status conv_wgrad_group(int n, const int (*shape)[5], const void* const* x,
                           const void* const* dy, float* const* dw, float* const* db,
                           void* const* ws, const size_t* ws_bytes, hipStream_t st) {
  if (n < 1 || n > sb::kWgMany) return SB_ERR_INVALID_ARG;
  sb::WgPlan p[sb::kWgMany];
  sb::WgArgs a[sb::kWgMany];
  int key = -2;
  for (int i = 0; i < n; ++i) {
    const int N = shape[i][0], C = shape[i][1], H = shape[i][2], W = shape[i][3],
              K = shape[i][4];
    const int k = conv_wgrad_batch_key(SB_F32, N, C, H, W, K, x[i], dy[i]);
    if (k < 0 || (key != -2 && k != key)) return SB_ERR_INVALID_ARG;
    key = k;
    const bool aligned = (((uintptr_t)x[i] | (uintptr_t)dy[i]) & 15) == 0;
    p[i] = sb::wg_plan(N, C, H, W, K, aligned, false);
    if (p[i].ws_bytes > 0 && (ws[i] == nullptr || ws_bytes[i] < p[i].ws_bytes))
      return SB_ERR_WORKSPACE;
    sb::WgArgs& g = a[i];
    g = sb::WgArgs{};
    g.x = x[i]; g.dy = dy[i]; g.dw = dw[i]; g.db = db ? db[i] : nullptr;
    g.part = p[i].splits > 1 ? (float*)ws[i] : nullptr;
    g.N = N; g.C = C; g.H = H; g.W = W; g.K = K;
    g.tiles_w = p[i].tiles_w; g.tiles_h = p[i].tiles_h; g.ptiles = p[i].ptiles;
    g.tiles_per_split = p[i].tps; g.c_tiles = p[i].c_tiles; g.splits = p[i].splits;
  }
  switch (key) {
    case 0: sb::wg_launch_many<sb::WgW32, float, false, false>(p, a, n, st); break;
    case 2: sb::wg_launch_many<sb::WgW32, float, true, false>(p, a, n, st); break;
    case 4: sb::wg_launch_many<sb::WgW16, float, false, false>(p, a, n, st); break;
    case 6: sb::wg_launch_many<sb::WgW16, float, true, false>(p, a, n, st); break;
    case 8: sb::wg_launch_many<sb::WgW8, float, false, false>(p, a, n, st); break;
    case 10: sb::wg_launch_many<sb::WgW8, float, true, false>(p, a, n, st); break;
    case 11: sb::wg_launch_many<sb::WgW8, float, true, true>(p, a, n, st); break;
    default: return SB_ERR_INVALID_ARG;
  }
  return launch_status();
}

// Channel-blocked bf16 tensors (SB_NCHW8C): the plan of the NCHW bf16 path
// (tiles of 64 pixels, 16 or 32 channels per block), the transpose-load
// kernel.
template <class T>
static void wg_launch_c8(const sb::WgPlan& p, const sb::WgArgs& a, hipStream_t st) {
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute((const void*)sb::conv3x3_wgrad_c8<T>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
  });
  dim3 grid(p.k_tiles * p.c_tiles, 1, p.splits);
  sb::conv3x3_wgrad_c8<T><<<grid, 256, T::LDS_BYTES, st>>>(a);
  if (p.splits > 1) sb::launch_splits_reduce(a.part, p.splits, a.K, a.C, a.dw, a.db, st);
}

bool conv_wgrad_c8_takes(int N, int C, int H, int W, int K) {
  return W >= 8 && C % 8 == 0 && K % 8 == 0 && sb::wg_plan(N, C, H, W, K, false, true).bc != 0;
}

size_t conv_wgrad_c8_ws(int N, int C, int H, int W, int K) {
  return sb::wg_plan(N, C, H, W, K, false, true).ws_bytes;
}

int conv_wgrad_c8_describe(int N, int C, int H, int W, int K, char* buf, size_t len) {
  sb::WgPlan p = sb::wg_plan(N, C, H, W, K, false, true);
  static const char* kT[] = {"2, 32", "4, 16", "8, 8"};
  return snprintf(buf, len, "sb::conv3x3_wgrad_c8<sb::WgC8Tile<%s, %d>> grid=%dx1x%d",
                  kT[p.tile], p.bc, p.k_tiles * p.c_tiles, p.splits);
}

sb_status conv_wgrad_c8(int N, int C, int H, int W, int K, const void* x, const void* dy,
                        float* dw, float* db, void* ws, size_t ws_bytes, hipStream_t st) {
  sb::WgPlan p = sb::wg_plan(N, C, H, W, K, false, true);
  if (!conv_wgrad_c8_takes(N, C, H, W, K)) return SB_ERR_UNSUPPORTED;
  if ((int64_t)std::max(C, K) * H * W * 2 >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  if (p.ws_bytes > 0 && (ws == nullptr || ws_bytes < p.ws_bytes)) return SB_ERR_WORKSPACE;
  sb::WgArgs a{};
  a.x = x; a.dy = dy; a.dw = dw; a.db = db;
  a.part = p.splits > 1 ? (float*)ws : nullptr;
  a.N = N; a.C = C; a.H = H; a.W = W; a.K = K;
  a.tiles_w = p.tiles_w; a.tiles_h = p.tiles_h; a.ptiles = p.ptiles;
  a.tiles_per_split = p.tps; a.c_tiles = p.c_tiles; a.splits = p.splits;
  if (p.bc == 32) {
    switch (p.tile) {
      case 0: wg_launch_c8<sb::WgC8Tile<2, 32, 32>>(p, a, st); break;
      case 1: wg_launch_c8<sb::WgC8Tile<4, 16, 32>>(p, a, st); break;
      default: wg_launch_c8<sb::WgC8Tile<8, 8, 32>>(p, a, st); break;
    }
  } else {
    switch (p.tile) {
      case 0: wg_launch_c8<sb::WgC8Tile<2, 32, 16>>(p, a, st); break;
      case 1: wg_launch_c8<sb::WgC8Tile<4, 16, 16>>(p, a, st); break;
      default: wg_launch_c8<sb::WgC8Tile<8, 8, 16>>(p, a, st); break;
    }
  }
  return launch_status();
}

}  // namespace sbh
