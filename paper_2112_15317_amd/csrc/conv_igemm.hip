// conv_igemm.hip -- 3x3 / stride 1 / pad 1 convolution forward and data
// gradient as an implicit GEMM on fp32 MFMA (v_mfma_f32_16x16x4_f32).
//
// Forward (sec. 2.2): out[n,co,h,w] = sum_{ci,r,s} in[n,ci,h+r-1,w+s-1] * w[co,ci,r,s].
// The data gradient is the same contraction with the filters transposed
// (co <-> ci) and rotated by 180 degrees: dx[n,c,i,j] = sum_{k,r,s}
// dy[n,k,i+r-1,j+s-1] * w[k,c,2-r,2-s].  Each kernel serves both; only the
// filter gather differs.
//
// Two kernels:
//
// conv3x3_igemm_f32 (any shape).  GEMM view per block: rows = BN output
// channels, columns = BM = 128 output pixels (IMGS images x TH rows x TW
// cols), reduction = input channels x 9 taps.  Per chunk of CK input
// channels the block stages in LDS the input halo (CK x IMGS x (TH+2) x
// (TW+2), read once, then read at 9 shifted windows: no im2col) and the
// filter slice [tap][ci][co].  Pipeline per chunk t: store chunk t+1 (already
// in registers) into the other LDS buffer, issue the global loads of chunk
// t+2, multiply chunk t out of LDS, barrier (the two-group 8x8 tiles do the
// store and the loads halfway through the multiply).  MFMA operand fragments are
// double-buffered in registers so LDS reads run one k-step ahead of the
// MFMAs.  Gathers are branch-free (clamped index + select).  MFMA rows are
// channels and columns pixels, so the 16 lanes of an output row store 16
// consecutive pixels (coalesced NCHW).
//
// conv3x3_small_f32 (whole images of 2x2 or 4x4 pixels, the late VGG
// layers).  A tile holds 16*G whole images, ordered position-major: one MFMA
// column block is 16 images at the same pixel position, so whether a tap
// falls in the zero padding is known at compile time for every block and
// those MFMAs are never issued (4 of 9 taps survive at 2x2, 100 of 144 at
// 4x4).  Whole images need no halo; LDS holds [ci][position][image] with the
// image index innermost (conflict-free operand reads), filled with float4
// loads of whole image planes.  The output tile is staged through LDS so it
// is written with coalesced float4 stores.
//
// conv3x3_few_f32 (passes with at most 4 output channels: the first layer's
// data gradient, whose outputs are the image's 3 channels).  An MFMA tile
// pads the output channels to at least 16 rows, so 3 channels would use
// 3/16 of its work; here each lane computes every output channel of 2
// vertically adjacent pixels on the vector ALU.  Per 8-channel chunk the
// block stages the input halo in LDS and the first 4 output channels of the
// packed filter slice (the 16-channel-output tile's slice, so packed buffers
// serve either kernel); a lane reads its 4 x 3 input neighbourhood of a
// channel once and each (tap, channel)'s filter values as one 16-byte LDS
// read at the same address in every lane.  (Scalar loads of the filter
// values straight into scalar registers measured slower: their latency sat
// in the FMA chain.)  Two groups of lanes split the channel chunks and add
// their sums at the end, in a fixed order.  The whole reduction runs in the
// block (no split).
//
// Both MFMA kernels split the channel chunks over gridDim.z when the output grid
// alone cannot fill the 256 CUs; each split writes its raw partial tile to
// the workspace and conv_splitk_reduce adds the splits in a fixed order and
// applies the epilogue.  (Reducing inside the kernel with a last-block
// counter needs device-scope fences, which write back the per-XCD L2s on
// this chip and cost far more than the extra launch.)
#include "conv_common.hpp"

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <type_traits>

namespace sb {

// ----------------------------------------------------------------- generic --
template <int TH_, int TW_, int IMGS_, int CK_, int BN_, int WAVES_N_, int KSPLIT_ = 1,
          int STAGED_ = 0>
struct ConvTile {
  static constexpr int TH = TH_, TW = TW_, IMGS = IMGS_, CK = CK_, BN = BN_;
  // STAGED: the unsplit output tile goes out through LDS ([channel][pixel])
  // in 16-byte pieces of 4 pixels of one row (full-row coalesced stores,
  // the mask read in the same pieces), instead of one 4-byte store per
  // accumulator element (16 lanes = 64 contiguous bytes).  For memory-bound
  // layers whose short channel loop leaves the epilogue a large share.
  static constexpr bool STAGED = STAGED_ != 0;
  // KSPLIT groups of 256 threads share the block's output tile and take
  // alternate channel chunks, each through its own LDS buffers; the groups'
  // partial sums are added through LDS in a fixed order at the end.  This
  // fills the chip on small grids without split partials in HBM.
  static constexpr int KSPLIT = KSPLIT_, THREADS = 256 * KSPLIT;
  static constexpr int BM = IMGS * TH * TW;
  static_assert(BM == 128 || BM == 256, "pixel tile must hold 128 or 256 pixels");
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
  static constexpr int LDS_X = CK * PLANE_P;
  static constexpr int LDS_W = 9 * CK * BN_P;
  // Halo staging lanes past the end of the halo store into a private slot
  // after the two regions (256 floats), so every halo staging store is
  // unconditional (no exec-mask juggling in the loop).
  static constexpr int LDS_SPARE = 256;
  static constexpr int LDS_BUF = LDS_X + LDS_W + LDS_SPARE;
  static constexpr size_t LDS_BYTES = KSPLIT * 2 * LDS_BUF * sizeof(float);
  static_assert(LDS_BYTES * (KSPLIT == 1 ? 2 : 1) <= 160 * 1024,
                "two blocks (one for KSPLIT = 2) must fit in the 160 KB of LDS");
  // Waves split the tile WAVES_N along channels x WAVES_M along pixels; a
  // wave owns WN channels x WM pixels (NB x MB MFMA blocks).  The 256-pixel
  // tiles give each wave 64 x 64, which halves the LDS operand reads per
  // MFMA and the filter staging per MFMA against 32 x 64.
  static constexpr int WAVES_N = WAVES_N_, WAVES_M = 4 / WAVES_N;
  static constexpr int WN = BN / WAVES_N, WM = BM / WAVES_M;
  static_assert(WN % 16 == 0 && WM % 16 == 0, "whole 16 x 16 MFMA blocks per wave");
  static constexpr int NB = WN / 16, MB = WM / 16;
  static constexpr int NSTEP = 9 * (CK / 4);     // MFMA k-steps per chunk
  // Halo layout per channel: [halo row][halo column][image], image
  // innermost, so that the 16 pixels of an MFMA column block (16 images, or
  // a row segment of several images) are 16 consecutive LDS words for every
  // tap: conflict-free operand reads however narrow the images.
  __host__ __device__ static constexpr int hoff(int img, int hy, int hx) {
    return (hy * HW + hx) * IMGS + img;
  }
  // Tile pixel p -> (image, row, column), in the same image-innermost order.
  __device__ static void pix(int p, int& img, int& yy, int& xx) {
    img = p % IMGS;
    const int q = p / IMGS;
    yy = q / TW;
    xx = q - yy * TW;
  }
};

// Whether MFMA column block mb of a wave at pixel-row position wm only
// multiplies zero padding at tap `tap`, when a tile spans the whole image
// height (H = TH): a 16-pixel column block lies in one tile row, and a tap
// in the top (bottom) filter row reads the padding row above (below) the
// image for the image's first (last) row.  Known at compile time after
// unrolling, so those MFMAs are never issued.
template <class T, bool WHOLE_H>
__device__ constexpr bool igemm_pad_block(int wm, int mb, int tap) {
  if (!WHOLE_H) return false;
  const int yy = (wm * T::WM + mb * 16) / T::IMGS / T::TW;
  return (tap / 3 == 0 && yy == 0) || (tap / 3 == 2 && yy == T::TH - 1);
}

// WHOLE_H: every tile spans the whole image height (H = TH); the MFMAs of
// column blocks whose taps read only padding rows are skipped.
// POOL (forward of fp32 tensors, unsplit, staged tiles): the output tile is
// not written; ReLU and 2x2 max pooling run on it in LDS (bias added: the
// tensor the unfused forward would write), and the pooled tile and its
// window codes go out instead (a.out, a.pool_idx), as sb_relu_maxpool_fwd
// computes them from that tensor.
template <class T, bool DGRAD, class E, bool WHOLE_H = false, bool POOL = false>
__global__ __launch_bounds__(T::THREADS, 2 / T::KSPLIT) void conv3x3_igemm_f32(ConvArgs a) {
  static_assert(!WHOLE_H || (T::TW * T::IMGS) % 16 == 0,
                "column blocks must not straddle tile rows");
  static_assert(!POOL || (!DGRAD && T::STAGED && std::is_same<E, float>::value &&
                          T::TH % 2 == 0 && T::TW % 2 == 0),
                "pooling: fp32 forward, staged tiles of whole 2x2 windows");
  extern __shared__ float lds_all[];

  // grp: which chunk stream this thread's 256-thread group takes.
  const int grp = threadIdx.x >> 8;
  float* lds = lds_all + grp * 2 * T::LDS_BUF;
  const int tid = threadIdx.x & 255, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % T::WAVES_M, wn = wave / T::WAVES_M;
  const int kq = lane >> 4, lr = lane & 15;

  int bt = blockIdx.x;
  const int tx = bt % a.tiles_w; bt /= a.tiles_w;
  const int ty = bt % a.tiles_h;
  const int tn = bt / a.tiles_h;
  const int n0 = tn * T::IMGS, h0 = ty * T::TH, w0 = tx * T::TW;
  const int co0 = blockIdx.y * T::BN;
  const int nchunks = cdiv(a.Cin, T::CK);
  const int kc0 = blockIdx.z * a.chunks_per_split;
  const int kc1 = min(nchunks, kc0 + a.chunks_per_split);
  const int HWs = a.H * a.W;

  // ---- gather plans (independent of the chunk) ----
  int x_off[T::HALO_PT], x_c[T::HALO_PT], x_loff[T::HALO_PT];
#pragma unroll
  for (int i = 0; i < T::HALO_PT; ++i) {
    int e = tid + i * 256;
    bool live = e < T::HALO;
    int c = e / T::PLANE, rem = e - c * T::PLANE;
    int img = rem % T::IMGS, q = rem / T::IMGS;          // rem = hoff(img, yy, xx)
    int yy = q / T::HW, xx = q - yy * T::HW;
    int n = n0 + img, h = h0 + yy - 1, w = w0 + xx - 1;
    bool ok = live && n < a.N && h >= 0 && h < a.H && w >= 0 && w < a.W;
    x_off[i] = ok ? img * a.Cin * HWs + h * a.W + w : -1;   // from image n0; + ci * H*W
    x_c[i] = c;
    x_loff[i] = live ? c * T::PLANE_P + rem : T::LDS_X + T::LDS_W + tid;
  }
  // Packed filter slice, 4 elements (one row, 4 consecutive columns) per
  // load: piece g = elements 4g .. 4g+3 -> LDS row 4g / BN, column 4g % BN.
  static_assert(T::BN % 4 == 0 && T::WTS % 4 == 0, "whole 4-column pieces");
  constexpr int WTS4 = T::WTS / 4, W4_PT = (WTS4 + 255) / 256;
  int w_loff[W4_PT];
#pragma unroll
  for (int i = 0; i < W4_PT; ++i) {
    const int e = 4 * (tid + i * 256);
    w_loff[i] = (e / T::BN) * T::BN_P + e % T::BN;
  }
  int pix_off[T::MB];
#pragma unroll
  for (int mb = 0; mb < T::MB; ++mb) {
    int img, yy, xx;
    T::pix(wm * T::WM + mb * 16 + lr, img, yy, xx);
    pix_off[mb] = T::hoff(img, yy, xx);
  }

  f4 acc[T::NB][T::MB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i)
#pragma unroll
    for (int j = 0; j < T::MB; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  const rsrc_t xr = input_rsrc<E>(a, n0, T::IMGS);
  const rsrc_t wr = packed_rsrc<E, T::WTS>(a, blockIdx.y);
  float rx[T::HALO_PT];
  f4 rw[W4_PT];
  auto gload = [&](int kc) {
    const int cbase = kc * T::CK;
#pragma unroll
    for (int i = 0; i < T::HALO_PT; ++i) {
      const int ci = cbase + x_c[i];
      const bool ok = x_off[i] >= 0 && ci < a.Cin;
      rx[i] = BufLoad<E>::one(xr, ok ? (uint32_t)(x_off[i] + ci * HWs) * (uint32_t)sizeof(E) : kOOB);
    }
#pragma unroll
    for (int i = 0; i < W4_PT; ++i) {
      const int g = tid + i * 256;
      rw[i] = BufLoad<E>::four(wr, g < WTS4 ? (uint32_t)(kc * T::WTS + 4 * g) * (uint32_t)sizeof(E)
                                            : kOOB);
    }
  };
  auto lstore = [&](int buf) {
    float* X = lds + buf * T::LDS_BUF;
    float* Wl = X + T::LDS_X;
#pragma unroll
    for (int i = 0; i < T::HALO_PT; ++i) X[x_loff[i]] = rx[i];
#pragma unroll
    for (int i = 0; i < W4_PT; ++i)
      if (WTS4 % 256 == 0 || tid + i * 256 < WTS4)
        *reinterpret_cast<f4*>(Wl + w_loff[i]) = rw[i];
  };
  // WMC: the wave's pixel-row position wm as a compile-time constant (only
  // used with WHOLE_H, to skip padding blocks).
  // mid(): staged at step MID of the chunk's MFMA sequence (the next
  // chunk's LDS store and the one after's global loads).  The two-group
  // 8x8 tiles stage halfway through, so the wait for the loads and the LDS
  // stores hide behind MFMAs; the other tiles stage before the first step.
  constexpr int MID = T::KSPLIT == 2 ? T::NSTEP / 2 : 0;
  auto compute_wm = [&](int buf, auto WMC, auto&& mid) {
    constexpr int WMc = decltype(WMC)::value;
    const float* X = lds + buf * T::LDS_BUF;
    const float* Wl = X + T::LDS_X;
    float fa[2][T::NB], fb[2][T::MB];
    auto frag = [&](int step, int slot) {
      const int tap = step / (T::CK / 4), cg = step - tap * (T::CK / 4);
      const int toff = T::hoff(0, tap / 3, tap % 3);
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
        fa[slot][nb] = Wl[(tap * T::CK + cg * 4 + kq) * T::BN_P + wn * T::WN + nb * 16 + lr];
#pragma unroll
      for (int mb = 0; mb < T::MB; ++mb)
        fb[slot][mb] = igemm_pad_block<T, WHOLE_H>(WMc, mb, tap)
                           ? 0.f : X[(cg * 4 + kq) * T::PLANE_P + pix_off[mb] + toff];
    };
    frag(0, 0);
#pragma unroll
    for (int s = 0; s < T::NSTEP; ++s) {
      if (s == MID) mid();
      if (s + 1 < T::NSTEP) frag(s + 1, (s + 1) & 1);
      const int tap = s / (T::CK / 4);
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb)
          if (!igemm_pad_block<T, WHOLE_H>(WMc, mb, tap))
            acc[nb][mb] = mfma16x16x4(fa[s & 1][nb], fb[s & 1][mb], acc[nb][mb]);
    }
  };
  auto compute = [&](int buf, auto&& mid) {
    if constexpr (WHOLE_H) {
      static_assert(T::WAVES_M <= 4, "at most four pixel-row positions");
      if (wm == 0) compute_wm(buf, std::integral_constant<int, 0>{}, mid);
      else if (T::WAVES_M > 1 && wm == 1) compute_wm(buf, std::integral_constant<int, 1>{}, mid);
      else if (T::WAVES_M > 2 && wm == 2) compute_wm(buf, std::integral_constant<int, 2>{}, mid);
      else if (T::WAVES_M > 3) compute_wm(buf, std::integral_constant<int, 3>{}, mid);
    } else {
      compute_wm(buf, std::integral_constant<int, 0>{}, mid);
    }
  };

  // Group g takes chunks kc0 + g, kc0 + g + KSPLIT, ...; every group runs the
  // same number of iterations (barriers are block-wide).
  const int nk = (kc1 - kc0 - grp + T::KSPLIT - 1) / T::KSPLIT;
  const int nit = (kc1 - kc0 + T::KSPLIT - 1) / T::KSPLIT;
  auto chunk = [&](int t) { return kc0 + grp + t * T::KSPLIT; };
  if (nk > 0) {
    gload(chunk(0));
    lstore(0);
    if (nk > 1) gload(chunk(1));
  }
  __syncthreads();
  for (int t = 0; t < nit; ++t) {
    const int buf = t & 1;
    // Buffer buf ^ 1 was last read before the previous barrier, so its next
    // contents may be stored at any point of this iteration.
    auto mid = [&]() {
      if (t + 1 < nk) lstore(buf ^ 1);
      if (t + 2 < nk) gload(chunk(t + 2));
    };
    if (t < nk) compute(buf, mid);
    else mid();
    __syncthreads();
  }

  if constexpr (T::KSPLIT == 2) {
    // Group 1 hands its partial tile to group 0 through LDS (lane-major, so
    // both the writes and the reads are conflict-free), group 0 adds it.
    constexpr int NACC = T::NB * T::MB;
    static_assert(4 * 64 * 4 * NACC <= 2 * T::LDS_BUF, "partial tile fits group 0's buffers");
    float* xfer = lds_all + (size_t)(wave * NACC * 4) * 64 + lane;
    if (grp == 1) {
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) xfer[((nb * T::MB + mb) * 4 + i) * 64] = acc[nb][mb][i];
    }
    __syncthreads();
    if (grp == 1) {
      // Without the staged output group 1 is done; with it, it still takes
      // part in the barriers and the stores below.
      if constexpr (!T::STAGED) return;
    } else {
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[nb][mb][i] += xfer[((nb * T::MB + mb) * 4 + i) * 64];
    }
  }

  // ---- epilogue: acc[nb][mb] lane holds channel co0 + wn*WN + nb*16 + 4*kq + i
  // of pixel wm*WM + mb*16 + lr ----
  const size_t total = (size_t)a.N * a.Cout * HWs;
  auto for_each_out = [&](auto&& fn) {
#pragma unroll
    for (int mb = 0; mb < T::MB; ++mb) {
      int img, yy, xx;
      T::pix(wm * T::WM + mb * 16 + lr, img, yy, xx);
      int n = n0 + img, h = h0 + yy, w = w0 + xx;
      if (n >= a.N || h >= a.H || w >= a.W) continue;
#pragma unroll
      for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int co = co0 + wn * T::WN + nb * 16 + kq * 4 + i;
          if (co >= a.Cout) continue;
          fn(acc[nb][mb][i], co, ((size_t)n * a.Cout + co) * HWs + (size_t)h * a.W + w);
        }
    }
  };
  if constexpr (T::STAGED) {
    // Output tile in LDS as [channel][image][row][column] (image-major, so
    // 4 consecutive tile columns are 4 consecutive image columns).
    static_assert(T::TW % 4 == 0, "4-pixel pieces within a tile row");
    constexpr int EP = T::BM + 4;                    // LDS row pitch: 4 mod 64 banks
    static_assert(T::BN * EP <= 2 * T::LDS_BUF, "output tile fits the LDS buffers");
    if (a.splits == 1) {
      // With one group every wave has passed the loop's last barrier; with
      // two, group 0 has just read the transfer area.
      if constexpr (T::KSPLIT == 2) __syncthreads();
      if (grp == 0) {
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb) {
          int img, yy, xx;
          T::pix(wm * T::WM + mb * 16 + lr, img, yy, xx);
          const int lp = (img * T::TH + yy) * T::TW + xx;
#pragma unroll
          for (int nb = 0; nb < T::NB; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              lds_all[(wn * T::WN + nb * 16 + kq * 4 + i) * EP + lp] = acc[nb][mb][i];
        }
      }
      __syncthreads();
      if constexpr (POOL) {
        // Pooled pixel q = (channel, image, pooled row, pooled column),
        // pooled columns fastest: per channel the first maximum in row-major
        // window order wins (strict >), the output is the maximum if it is
        // positive, else +0, and bit 7 of the code flags the latter.
        constexpr int PTH = T::TH / 2, PTW = T::TW / 2, PP = T::IMGS * PTH * PTW;
        static_assert(T::BN * PP % T::THREADS == 0, "whole rounds of pooled pixels");
        const int Hh = a.H / 2, Wh = a.W / 2;
#pragma unroll 4
        for (int j = 0; j < T::BN * PP / T::THREADS; ++j) {
          const int q = (int)threadIdx.x + T::THREADS * j;
          const int col = q / PP, pp = q % PP;
          const int img = pp / (PTH * PTW), r = pp % (PTH * PTW);
          const int py = r / PTW, px = r % PTW;
          const int n = n0 + img, oh = h0 / 2 + py, ow = w0 / 2 + px, co = co0 + col;
          if (n >= a.N || oh >= Hh || ow >= Wh || co >= a.Cout) continue;
          const float* l = lds_all + col * EP + (img * T::TH + 2 * py) * T::TW + 2 * px;
          const float bv = a.bias ? a.bias[co] : 0.f;
          const float v[4] = {l[0] + bv, l[1] + bv, l[T::TW] + bv, l[T::TW + 1] + bv};
          float m = v[0];
          uint32_t c = 0;
#pragma unroll
          for (int k = 1; k < 4; ++k)
            if (v[k] > m) { m = v[k]; c = (uint32_t)k; }
          const bool pos = m > 0.f;
          const size_t off = (((size_t)n * a.Cout + co) * Hh + oh) * Wh + ow;
          ((float*)a.out)[off] = pos ? m : 0.f;
          a.pool_idx[off] = (uint8_t)(c | (pos ? 0u : 0x80u));
        }
        return;
      }
      constexpr int QPR = T::BM / 4;                 // 4-pixel pieces per channel row
      static_assert(T::BN * QPR % T::THREADS == 0, "whole rounds of pieces");
      const bool vec = std::is_same<E, float>::value && a.W % 4 == 0 &&
                       (((uintptr_t)a.out | (uintptr_t)a.mask) & 15) == 0;
#pragma unroll
      for (int j = 0; j < T::BN * QPR / T::THREADS; ++j) {
        const int q = (int)threadIdx.x + T::THREADS * j;
        const int col = q / QPR, px = (q % QPR) * 4;
        const int img = px / (T::TH * T::TW), rem = px % (T::TH * T::TW);
        const int co = co0 + col, h = h0 + rem / T::TW, w = w0 + rem % T::TW;
        if (co >= a.Cout || n0 + img >= a.N || h >= a.H || w >= a.W) continue;
        const f4 v = *reinterpret_cast<const f4*>(lds_all + col * EP + px);
        const size_t off = ((size_t)(n0 + img) * a.Cout + co) * HWs + (size_t)h * a.W + w;
        if (vec) {
          const float bv = a.bias ? a.bias[co] : 0.f;
          f4 mk = f4{1.f, 1.f, 1.f, 1.f};
          if (a.mask) mk = *reinterpret_cast<const f4*>((const float*)a.mask + off);
          f4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float r = v[e] + bv;
            if (a.relu && !(r > 0.f)) r = 0.f;
            o[e] = mk[e] > 0.f ? r : 0.f;
          }
          *reinterpret_cast<f4*>((float*)a.out + off) = o;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (w + e < a.W)
              Elem<E>::store((E*)a.out, off + e, conv_epilogue<E>(a, v[e], co, off + e));
        }
      }
      return;
    }
  }
  if constexpr (T::KSPLIT == 2 && T::STAGED) {
    if (grp == 1) return;                            // split partials: group 0 writes them
  }
  if (a.splits == 1) {
    for_each_out([&](float v, int co, size_t off) {
      Elem<E>::store((E*)a.out, off, conv_epilogue<E>(a, v, co, off));
    });
    return;
  }
  float* mine = a.part + (size_t)blockIdx.z * total;
  for_each_out([&](float v, int, size_t off) { mine[off] = v; });
}

// ------------------------------------------------------ small whole images --
template <int H_, int W_, int G_, int KSPLIT_ = 1>
struct SmallTile {
  static constexpr int H = H_, W = W_, G = G_;
  // KSPLIT = 2: two groups of 256 threads take alternate channel chunks
  // through LDS buffers of their own and add their tiles in LDS at the end
  // (as the two-group 8x8 tiles): half the split partials in HBM for the
  // same number of resident waves.
  static constexpr int KSPLIT = KSPLIT_, THREADS = 256 * KSPLIT;
  static constexpr int P = H * W;                 // positions per image
  static constexpr int IMGS = 16 * G;             // images per tile
  static constexpr int BM = IMGS * P;             // pixels per tile
  static constexpr int CK = 8, BN = 64, BN_P = 80;
  // Channel plane in LDS: [position][image], position rows PS = IMGS + 1
  // apart.  The staging stores of a wave (4 positions x 8 channels x 2
  // images for the 4x4 tile) then spread over 32 banks instead of 8; the
  // operand reads (16 consecutive images of one row) stay conflict-free.
  static constexpr int PS = IMGS + 1;
  static constexpr int PLANE = P * PS;
  // Channel stride: the smallest >= PLANE that is 16 mod 64, so the four
  // k-rows of an operand read land in different banks.
  static constexpr int PLANE_P = (PLANE - 16 + 63) / 64 * 64 + 16;
  static constexpr int LDS_X = CK * PLANE_P;
  static constexpr int LDS_W = 9 * CK * BN_P;
  static constexpr int LDS_BUF = LDS_X + LDS_W;
  static_assert(P % 4 == 0, "image planes are loaded as float4");
  static constexpr int X_F4 = CK * IMGS * P / 4;  // float4 per chunk
  static constexpr int X_PT = X_F4 / 256;
  static constexpr int WTS = 9 * CK * BN;
  // Every image-plane staging lane is live: those stores need no condition.
  static_assert(X_F4 % 256 == 0 && WTS % 4 == 0, "staging covers whole 256-thread rounds");
  static constexpr int MB = BM / 16;              // column blocks: (position, image group)
  static constexpr int OUT_IMG_STRIDE = BN * P + 4;
  static constexpr int LDS_OUT = IMGS * OUT_IMG_STRIDE;
  static constexpr int LDS_FLOATS =
      KSPLIT * 2 * LDS_BUF > LDS_OUT ? KSPLIT * 2 * LDS_BUF : LDS_OUT;
  static constexpr size_t LDS_BYTES = LDS_FLOATS * sizeof(float);
  static_assert(LDS_BYTES * (KSPLIT == 1 ? 2 : 1) <= 160 * 1024,
                "two blocks (one for KSPLIT = 2) must fit in the 160 KB of LDS");
  // Source position of tap (r,s) at position pos, or -1 if it is padding.
  __host__ __device__ static constexpr int src(int pos, int tap) {
    return (pos / W + tap / 3 - 1 >= 0 && pos / W + tap / 3 - 1 < H &&
            pos % W + tap % 3 - 1 >= 0 && pos % W + tap % 3 - 1 < W)
               ? (pos / W + tap / 3 - 1) * W + (pos % W + tap % 3 - 1)
               : -1;
  }
};

template <class T, bool DGRAD, class E>
__global__ __launch_bounds__(T::THREADS, 2 / T::KSPLIT) void conv3x3_small_f32(ConvArgs a) {
  extern __shared__ float lds_all[];
  // grp: which chunk stream this thread's 256-thread group takes.
  const int grp = threadIdx.x >> 8;
  float* lds = lds_all + grp * 2 * T::LDS_BUF;
  const int tid = threadIdx.x & 255, lane = tid & 63, wave = tid >> 6;
  const int kq = lane >> 4, lr = lane & 15;
  const int n0 = blockIdx.x * T::IMGS;
  const int co0 = blockIdx.y * T::BN;
  const int nchunks = cdiv(a.Cin, T::CK);
  const int kc0 = blockIdx.z * a.chunks_per_split;
  const int kc1 = min(nchunks, kc0 + a.chunks_per_split);

  // Image planes: float4 q of the chunk = (image, channel, quarter), quarter
  // fastest: neighbouring threads read consecutive 16-byte pieces of one
  // image's channel planes, which are contiguous in NCHW (fully coalesced).
  int x_off[T::X_PT], x_c[T::X_PT], x_loff[T::X_PT];
#pragma unroll
  for (int i = 0; i < T::X_PT; ++i) {
    int q = tid + i * 256;
    int quarter = q % (T::P / 4), rest = q / (T::P / 4);
    int c = rest % T::CK, img = rest / T::CK;
    int n = n0 + img;
    x_off[i] = n < a.N ? img * a.Cin * T::P + quarter * 4 : -1;   // from image n0; + ci * P
    x_c[i] = c;
    x_loff[i] = c * T::PLANE_P + quarter * 4 * T::PS + img;
  }
  // Packed filter slice, 4 elements (one row, 4 consecutive columns) per
  // load: piece g = elements 4g .. 4g+3 -> LDS row 4g / BN, column 4g % BN.
  constexpr int WTS4 = T::WTS / 4, W4_PT = (WTS4 + 255) / 256;
  int w_loff[W4_PT];
#pragma unroll
  for (int i = 0; i < W4_PT; ++i) {
    const int e = 4 * (tid + i * 256);
    w_loff[i] = (e / T::BN) * T::BN_P + e % T::BN;
  }

  f4 acc[T::MB];
#pragma unroll
  for (int j = 0; j < T::MB; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};

  const rsrc_t xr = input_rsrc<E>(a, n0, T::IMGS);
  const rsrc_t wr = packed_rsrc<E, T::WTS>(a, blockIdx.y);
  f4 rx[T::X_PT];
  f4 rw[W4_PT];
  auto gload = [&](int kc) {
    const int cbase = kc * T::CK;
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) {
      const int ci = cbase + x_c[i];
      const bool ok = x_off[i] >= 0 && ci < a.Cin;
      rx[i] = BufLoad<E>::four(xr, ok ? (uint32_t)(x_off[i] + ci * T::P) * (uint32_t)sizeof(E) : kOOB);
    }
#pragma unroll
    for (int i = 0; i < W4_PT; ++i) {
      const int g = tid + i * 256;
      rw[i] = BufLoad<E>::four(wr, g < WTS4 ? (uint32_t)(kc * T::WTS + 4 * g) * (uint32_t)sizeof(E)
                                            : kOOB);
    }
  };
  auto lstore = [&](int buf) {
    float* X = lds + buf * T::LDS_BUF;
    float* Wl = X + T::LDS_X;
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) X[x_loff[i] + j * T::PS] = rx[i][j];
#pragma unroll
    for (int i = 0; i < W4_PT; ++i)
      if (WTS4 % 256 == 0 || tid + i * 256 < WTS4)
        *reinterpret_cast<f4*>(Wl + w_loff[i]) = rw[i];
  };
  auto compute = [&](int buf) {
    const float* X = lds + buf * T::LDS_BUF;
    const float* Wl = X + T::LDS_X;
#pragma unroll
    for (int tap = 0; tap < 9; ++tap)
#pragma unroll
      for (int cg = 0; cg < T::CK / 4; ++cg) {
        const float fa = Wl[(tap * T::CK + cg * 4 + kq) * T::BN_P + wave * 16 + lr];
#pragma unroll
        for (int mb = 0; mb < T::MB; ++mb) {
          const int pos = mb / T::G, g = mb % T::G;
          const int sp = T::src(pos, tap);
          if (sp < 0) continue;                       // padding: resolved at compile time
          const float fb = X[(cg * 4 + kq) * T::PLANE_P + sp * T::PS + g * 16 + lr];
          acc[mb] = mfma16x16x4(fa, fb, acc[mb]);
        }
      }
  };

  // Group g takes chunks kc0 + g, kc0 + g + KSPLIT, ...; every group runs
  // the same number of iterations (barriers are block-wide).
  const int nk = (kc1 - kc0 - grp + T::KSPLIT - 1) / T::KSPLIT;
  const int nit = (kc1 - kc0 + T::KSPLIT - 1) / T::KSPLIT;
  auto chunk = [&](int t) { return kc0 + grp + t * T::KSPLIT; };
  if (nk > 0) {
    gload(chunk(0));
    lstore(0);
    if (nk > 1) gload(chunk(1));
  }
  __syncthreads();
  for (int t = 0; t < nit; ++t) {
    const int buf = t & 1;
    if (t + 1 < nk) lstore(buf ^ 1);
    if (t + 2 < nk) gload(chunk(t + 2));
    if (t < nk) compute(buf);
    __syncthreads();
  }
  if constexpr (T::KSPLIT == 2) {
    // Group 1 hands its tile to group 0 through LDS (lane-major:
    // conflict-free), group 0 adds it; both then take part in the staging
    // barrier below, and group 1 leaves before the stores.
    static_assert(4 * 64 * 4 * T::MB <= T::LDS_FLOATS, "partial tile fits the LDS");
    float* xfer = lds_all + (size_t)(wave * T::MB * 4) * 64 + lane;
    if (grp == 1) {
#pragma unroll
      for (int mb = 0; mb < T::MB; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) xfer[(mb * 4 + i) * 64] = acc[mb][i];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int mb = 0; mb < T::MB; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[mb][i] += xfer[(mb * 4 + i) * 64];
    }
    __syncthreads();
  }

  // Stage the tile as [image][channel][position] so rows of the output go
  // out as float4 stores.  acc[mb] lane holds channel wave*16 + 4*kq + i of
  // image g*16 + lr at position pos (mb = pos*G + g).
  if (grp == 0) {
#pragma unroll
    for (int mb = 0; mb < T::MB; ++mb) {
      const int pos = mb / T::G, g = mb % T::G;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        lds_all[(g * 16 + lr) * T::OUT_IMG_STRIDE + (wave * 16 + kq * 4 + i) * T::P + pos] =
            acc[mb][i];
    }
  }
  __syncthreads();
  if (grp != 0) return;
  // The tile's output: for each image, channels [co0, co0+BN) x P positions
  // are contiguous in NCHW.  float4 q -> (image, channel, quarter).
  constexpr int OUT_F4 = T::IMGS * T::BN * T::P / 4;
  const size_t total = (size_t)a.N * a.Cout * T::P;
  auto for_each_out4 = [&](auto&& fn) {
    for (int q = tid; q < OUT_F4; q += 256) {
      int quarter = q % (T::P / 4), rest = q / (T::P / 4);
      int cl = rest % T::BN, img = rest / T::BN;
      int n = n0 + img, co = co0 + cl;
      if (n >= a.N || co >= a.Cout) continue;
      const float* s = lds + img * T::OUT_IMG_STRIDE + cl * T::P + quarter * 4;
      f4 v = {s[0], s[1], s[2], s[3]};
      fn(v, co, ((size_t)n * a.Cout + co) * T::P + quarter * 4);
    }
  };
  auto epi4 = [&](f4 v, int co, size_t off) {
    f4 m = {1.f, 1.f, 1.f, 1.f};
    if (a.mask) m = Elem<E>::load4((const E*)a.mask + off);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float x = v[j];
      if (a.bias) x += a.bias[co];
      if (a.relu && !(x > 0.f)) x = 0.f;
      if (a.mask && !(m[j] > 0.f)) x = 0.f;
      v[j] = x;
    }
    Elem<E>::store4((E*)a.out + off, v);
  };
  if (a.splits == 1) {
    for_each_out4(epi4);
    return;
  }
  float* mine = a.part + (size_t)blockIdx.z * total;
  for_each_out4([&](f4 v, int, size_t off) { *reinterpret_cast<f4*>(mine + off) = v; });
}

// ------------------------------------------------- few output channels --
struct FewTile {
  static constexpr int TH = 8, TW = 32, CK = 8, BN = 16;   // BN: the packed slice's width
  // Two groups of 128 lanes (2 pixels, rows, per lane) take alternate
  // channel chunks through LDS buffers of their own and add their sums in
  // LDS at the end: two waves per SIMD for the grid's one wave per SIMD of
  // pixels.
  static constexpr int GT = 128, THREADS = 2 * GT;
  static constexpr int HH = TH + 2, HW = TW + 2, PLANE = HH * HW;
  static constexpr int XS = CK * PLANE;                      // halo floats per chunk
  static constexpr int X_PT = (XS + GT - 1) / GT;
  static constexpr int WQ = 9 * CK;                          // (tap, channel) rows of 4
  static constexpr int W_PT = (WQ * 4 + GT - 1) / GT;
};

template <int CO, class E>
__global__ __launch_bounds__(FewTile::THREADS) void conv3x3_few_f32(ConvArgs a) {
  using T = FewTile;
  static_assert(CO >= 1 && CO <= 4, "one 16-byte filter read per (tap, channel)");
  static_assert(T::GT * 2 * CO <= 2 * T::XS, "the partial sums fit one group's halo buffers");
  __shared__ float X[2][2][T::XS];                 // [group][buffer]
  __shared__ f4 Wl[2][2][T::WQ];
  const int grp = threadIdx.x / T::GT, tid = threadIdx.x % T::GT;
  const int tx = tid % T::TW, ty = (tid / T::TW) * 2;   // the lane's pixels: rows ty, ty + 1
  int bt = blockIdx.x;
  const int txi = bt % a.tiles_w; bt /= a.tiles_w;
  const int tyi = bt % a.tiles_h;
  const int n = bt / a.tiles_h;
  const int h0 = tyi * T::TH, w0 = txi * T::TW;
  const int HWs = a.H * a.W;
  const int nchunks = cdiv(a.Cin, T::CK);
  // Raw buffer loads: out-of-range offsets read 0.  Padding offsets start at
  // kOOB and the channels past Cin in the last chunk lie past the image's
  // range, so adding a chunk's offset keeps both out of range.
  const rsrc_t xr = input_rsrc<E>(a, n, 1);
  const rsrc_t wr = packed_rsrc<E, 9 * T::CK * T::BN>(a, 0);

  // Staging plan: halo element e = (channel, halo row, halo column); its
  // byte offset within the chunk.
  uint32_t x_off[T::X_PT];
#pragma unroll
  for (int i = 0; i < T::X_PT; ++i) {
    const int e = tid + i * T::GT;
    const int c = e / T::PLANE, r = e % T::PLANE;
    const int h = h0 + r / T::HW - 1, w = w0 + r % T::HW - 1;
    const bool ok = e < T::XS && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
    x_off[i] = ok ? (uint32_t)((c * HWs + h * a.W + w) * (int)sizeof(E)) : kOOB;
  }
  // Filter value f = (tap, channel) row f / 4, output channel f % 4 of the
  // chunk's packed slice [tap][channel][BN output channels].
  uint32_t w_off[T::W_PT];
#pragma unroll
  for (int i = 0; i < T::W_PT; ++i) {
    const int f = tid + i * T::GT;
    w_off[i] = f < T::WQ * 4 ? (uint32_t)(((f / 4) * T::BN + f % 4) * (int)sizeof(E)) : kOOB;
  }
  float rx[T::X_PT], rw[T::W_PT];
  auto gload = [&](int kc) {
    const uint32_t xc = (uint32_t)(kc * T::CK * HWs * (int)sizeof(E));
    const uint32_t wc = (uint32_t)(kc * T::WQ * T::BN * (int)sizeof(E));
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) rx[i] = BufLoad<E>::one(xr, x_off[i] + xc);
#pragma unroll
    for (int i = 0; i < T::W_PT; ++i) rw[i] = BufLoad<E>::one(wr, w_off[i] + wc);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < T::X_PT; ++i) {
      const int e = tid + i * T::GT;
      if (e < T::XS) X[grp][buf][e] = rx[i];
    }
#pragma unroll
    for (int i = 0; i < T::W_PT; ++i) {
      const int f = tid + i * T::GT;
      if (f < T::WQ * 4) reinterpret_cast<float*>(Wl[grp][buf])[f] = rw[i];
    }
  };

  float acc[2][CO];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int co = 0; co < CO; ++co) acc[q][co] = 0.f;
  auto compute = [&](int buf) {
    const float* Xb = X[grp][buf];
    const f4* Wb = Wl[grp][buf];
    // Two channels at a time: unrolling all eight would let the compiler
    // hoist every channel's reads and spill.
#pragma unroll 2
    for (int c = 0; c < T::CK; ++c) {
      // Halo rows ty .. ty + 3, columns tx .. tx + 2: both pixels' taps.
      float v[4][3];
#pragma unroll
      for (int dr = 0; dr < 4; ++dr)
#pragma unroll
        for (int ds = 0; ds < 3; ++ds) v[dr][ds] = Xb[c * T::PLANE + (ty + dr) * T::HW + tx + ds];
#pragma unroll
      for (int tap = 0; tap < 9; ++tap) {
        const f4 wv = Wb[tap * T::CK + c];       // the same address in every lane
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int co = 0; co < CO; ++co)
            acc[q][co] = fmaf(v[q + tap / 3][tap % 3], wv[co], acc[q][co]);
      }
    }
  };

  // Group g takes chunks g, g + 2, ...; both run the same number of
  // iterations (the barriers are block-wide).
  const int nit = (nchunks + 1) / 2;
  auto live = [&](int t) { return 2 * t + grp < nchunks; };
  if (live(0)) {
    gload(grp);
    lstore(0);
  }
  __syncthreads();
  for (int t = 0; t < nit; ++t) {
    const int buf = t & 1;
    if (live(t + 1)) gload(2 * (t + 1) + grp);
    if (live(t)) compute(buf);
    if (live(t + 1)) lstore(buf ^ 1);
    __syncthreads();
  }
  // Group 1 hands its sums to group 0 through its own halo buffers (lane
  // fastest: conflict-free), group 0 adds them and stores.
  float* xfer = &X[1][0][0];
  if (grp == 1) {
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int co = 0; co < CO; ++co) xfer[(q * CO + co) * T::GT + tid] = acc[q][co];
  }
  __syncthreads();
  if (grp == 1) return;
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int co = 0; co < CO; ++co) acc[q][co] += xfer[(q * CO + co) * T::GT + tid];

  const int j = w0 + tx;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int i = h0 + ty + q;
    if (i >= a.H || j >= a.W) continue;
#pragma unroll
    for (int co = 0; co < CO; ++co) {
      if (co >= a.Cout) continue;
      const size_t off = ((size_t)n * a.Cout + co) * HWs + (size_t)i * a.W + j;
      Elem<E>::store((E*)a.out, off, conv_epilogue<E>(a, acc[q][co], co, off));
    }
  }
}

// ---------------------------------------------------------------- host --
struct IgemmPlan {
  int tile;          // index into the tile table
  int imgs;          // images per pixel tile
  int grid_x, co_tiles;
  int tiles_w, tiles_h;
  int nchunks, cps, splits;
  size_t pack_bytes;  // packed filters, at the start of the workspace
  size_t part_off;    // split partials, after them
  size_t ws_bytes;
};

using TileW32 = ConvTile<4, 32, 1, 8, 64, 2, 1, 1>;
using TileW16 = ConvTile<8, 16, 1, 8, 64, 2, 1, 1>;
using TileW8 = ConvTile<8, 8, 2, 8, 64, 2, 1, 1>;
using TileW4 = ConvTile<4, 4, 8, 8, 64, 2>;
using TileW2 = ConvTile<2, 2, 32, 8, 64, 2>;
using TileW32c4 = ConvTile<4, 32, 1, 4, 64, 2, 1, 1>;   // output staged through LDS
using TileW32n16 = ConvTile<4, 32, 1, 8, 16, 1>;
using TileW32L = ConvTile<8, 32, 1, 8, 64, 1, 1, 1>;
using TileW16L = ConvTile<16, 16, 1, 8, 64, 1, 1, 1>;
using TileW8L = ConvTile<8, 8, 4, 8, 64, 1, 1, 1>;
using TileW8K2 = ConvTile<8, 8, 2, 8, 64, 2, 2, 1>;
using Small2 = SmallTile<2, 2, 2>;
using Small4 = SmallTile<4, 4, 1>;
using Small2K2 = SmallTile<2, 2, 2, 2>;
using Small4K2 = SmallTile<4, 4, 1, 2>;

static const char* kTileNames[] = {
    "sb::conv3x3_igemm_f32<sb::ConvTile<4, 32, 1, 8, 64, 2, 1, 1>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<8, 16, 1, 8, 64, 2, 1, 1>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<8, 8, 2, 8, 64, 2, 1, 1>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<4, 4, 8, 8, 64, 2, 1, 0>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<2, 2, 32, 8, 64, 2, 1, 0>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<4, 32, 1, 4, 64, 2, 1, 1>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<4, 32, 1, 8, 16, 1, 1, 0>, %s, %s>",
    "sb::conv3x3_small_f32<sb::SmallTile<2, 2, 2, 1>, %s, %s>",
    "sb::conv3x3_small_f32<sb::SmallTile<4, 4, 1, 1>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<8, 32, 1, 8, 64, 1, 1, 1>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<16, 16, 1, 8, 64, 1, 1, 1>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<8, 8, 4, 8, 64, 1, 1, 1>, %s, %s>",
    "sb::conv3x3_igemm_f32<sb::ConvTile<8, 8, 2, 8, 64, 2, 2, 1>, %s, %s>",
    "sb::conv3x3_small_f32<sb::SmallTile<2, 2, 2, 2>, %s, %s>",
    "sb::conv3x3_small_f32<sb::SmallTile<4, 4, 1, 2>, %s, %s>",
};

// allow_small: the whole-image kernel needs tensors aligned for 4-element
// moves.
static IgemmPlan igemm_plan(int N, int Cin, int H, int W, int Cout, int esize,
                            bool allow_small = true) {
  IgemmPlan p{};
  int th = 4, tw = 32, imgs = 1, ck = 8, bn = 64;
  if (allow_small && H == 2 && W == 2 && Cin > 4) { p.tile = 7; th = 2; tw = 2; imgs = 32; }
  else if (allow_small && H == 4 && W == 4 && Cin > 4) { p.tile = 8; th = 4; tw = 4; imgs = 16; }
  else if (Cout <= 16 && Cin > 4 && W >= 32) { p.tile = 6; bn = 16; }
  else if (Cin <= 4 && W >= 32) { p.tile = 5; ck = 4; }
  else if (W >= 32 && (long)N * cdiv(H, 8) * cdiv(W, 32) >= 512) { p.tile = 9; th = 8; }
  else if (W >= 32) { p.tile = 0; }
  else if (W >= 16) { p.tile = 1; th = 8; tw = 16; }
  else if (W >= 8) { p.tile = 2; th = 8; tw = 8; imgs = 2; }
  else if (W >= 4) { p.tile = 3; th = 4; tw = 4; imgs = 8; }
  else { p.tile = 4; th = 2; tw = 2; imgs = 32; }
  p.imgs = imgs;
  p.tiles_w = cdiv(W, tw);
  p.tiles_h = cdiv(H, th);
  p.grid_x = p.tiles_w * p.tiles_h * cdiv(N, imgs);
  p.co_tiles = cdiv(Cout, bn);
  p.nchunks = cdiv(Cin, ck);
  long blocks = (long)p.grid_x * p.co_tiles;
  // 8x8-image tiles that cannot fill the chip take the two-group block
  // (intra-block split over channel chunks) before any split in HBM.
  if (p.tile == 2 && blocks < 512 && p.nchunks >= 4) { p.tile = 12; blocks *= 2; }
  // Whole-image tiles likewise: two groups per block halve the split
  // partials written to and read back from HBM.
  if ((p.tile == 7 || p.tile == 8) && blocks < 512 && p.nchunks >= 4) {
    p.tile = p.tile == 7 ? 13 : 14;
    blocks *= 2;
  }
  // About two resident 256-thread groups on each of the 256 CUs; at most 8
  // splits, and at least two chunks per split.
  const long target = 512;
  int splits = 1;
  if (blocks < target)
    splits = (int)std::min<long>(std::min<long>(8, std::max(1, p.nchunks / 2)),
                                 cdiv((int)target, (int)blocks));
  p.cps = cdiv(p.nchunks, splits);
  p.splits = cdiv(p.nchunks, p.cps);
  p.pack_bytes = (size_t)p.co_tiles * p.nchunks * 9 * ck * bn * esize;
  p.part_off = round_up(p.pack_bytes, 256);
  p.ws_bytes = p.part_off +
               (p.splits > 1 ? (size_t)p.splits * N * Cout * H * W * sizeof(float) : 0);
  return p;
}

// pack: the call packs the filters itself (into the workspace); otherwise
// a.wpk already holds them.
// Tiles of 8x8 pixels (whole images of 8-row layers) have a variant that
// skips the MFMAs of padding rows.
template <class T, bool SMALL>
constexpr bool has_whole_h() {
  if constexpr (SMALL) return false;
  else return T::TH == 8 && T::TW == 8;
}

// Tiles whose forward can pool in its epilogue (fp32, staged output tile of
// whole 2x2 windows).
template <class T, bool SMALL, class E>
constexpr bool can_pool() {
  if constexpr (SMALL) return false;
  else return T::STAGED && std::is_same<E, float>::value && T::TH % 2 == 0 && T::TW % 2 == 0;
}

template <class T, bool DGRAD, bool SMALL, class E>
static void igemm_launch(const IgemmPlan& p, const ConvArgs& a, bool pack, hipStream_t st) {
  static bool attr_set = false;
  constexpr bool can_whole = has_whole_h<T, SMALL>();
  constexpr bool pool_ok = !DGRAD && can_pool<T, SMALL, E>();
  const bool whole = can_whole && a.H == 8;
  if (!attr_set) {
    if constexpr (SMALL) {
      (void)hipFuncSetAttribute((const void*)conv3x3_small_f32<T, DGRAD, E>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
    } else {
      (void)hipFuncSetAttribute((const void*)conv3x3_igemm_f32<T, DGRAD, E>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
      if constexpr (can_whole)
        (void)hipFuncSetAttribute((const void*)conv3x3_igemm_f32<T, DGRAD, E, true>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)T::LDS_BYTES);
      if constexpr (pool_ok) {
        (void)hipFuncSetAttribute((const void*)conv3x3_igemm_f32<T, false, E, false, true>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)T::LDS_BYTES);
        if constexpr (can_whole)
          (void)hipFuncSetAttribute((const void*)conv3x3_igemm_f32<T, false, E, true, true>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize,
                                    (int)T::LDS_BYTES);
      }
    }
    attr_set = true;
  }
  if (pack)
    filter_pack<DGRAD, T::CK, T::BN, E><<<p.co_tiles * p.nchunks, 256, 0, st>>>(
        (const E*)a.wt, (E*)a.wpk, a.Cin, a.Cout);
  dim3 grid(p.grid_x, p.co_tiles, p.splits);
  ConvArgs k = a;
  if (p.splits > 1) { k.bias = nullptr; k.mask = nullptr; k.relu = 0; }
  if (a.pool_idx && p.splits == 1) {       // the caller checked the plan can pool
    if constexpr (pool_ok) {
      if constexpr (can_whole) {
        if (whole) {
          conv3x3_igemm_f32<T, false, E, true, true><<<grid, T::THREADS, T::LDS_BYTES, st>>>(k);
          return;
        }
      }
      conv3x3_igemm_f32<T, false, E, false, true><<<grid, T::THREADS, T::LDS_BYTES, st>>>(k);
    }
    return;
  }
  if constexpr (SMALL) {
    conv3x3_small_f32<T, DGRAD, E><<<grid, T::THREADS, T::LDS_BYTES, st>>>(k);
  } else {
    if constexpr (can_whole) {
      if (whole) conv3x3_igemm_f32<T, DGRAD, E, true><<<grid, T::THREADS, T::LDS_BYTES, st>>>(k);
      else conv3x3_igemm_f32<T, DGRAD, E><<<grid, T::THREADS, T::LDS_BYTES, st>>>(k);
    } else {
      conv3x3_igemm_f32<T, DGRAD, E><<<grid, T::THREADS, T::LDS_BYTES, st>>>(k);
    }
  }
  if (p.splits > 1) {
    size_t total = (size_t)a.N * a.Cout * a.H * a.W;
    const unsigned pg = (unsigned)((total / 4 + 255) / 256);
    if (a.pool_idx && ((uintptr_t)a.part & 7) == 0)   // pooled forward: the reduction pools
      conv_splitk_reduce_pool<E, true><<<pg, 256, 0, st>>>(
          a.part, p.splits, total, a.Cout, a.H, a.W, a.bias, (E*)a.out, a.pool_idx);
    else if (a.pool_idx)
      conv_splitk_reduce_pool<E, false><<<pg, 256, 0, st>>>(
          a.part, p.splits, total, a.Cout, a.H, a.W, a.bias, (E*)a.out, a.pool_idx);
    else
      launch_splitk_reduce<E>(a.part, p.splits, total, a.Cout, a.H * a.W, a.bias, a.relu,
                              (const E*)a.mask, (E*)a.out, st);
  }
}

// Passes with at most 4 output channels on the 16-channel-output tile's plan
// (and its packed filters) take the vector-ALU kernel, in the whole
// reduction: 8 x 32-pixel tiles, no split.
inline bool few_takes(const IgemmPlan& p, int Cout) { return p.tile == 6 && Cout <= 4; }

// Whether an fp32 forward on plan p can pool in the call: a split plan
// pools in its split reduction; an unsplit one in its epilogue if its tile
// is staged and holds whole 2x2 windows (not the few-channel kernel).
inline bool igemm_pools(const IgemmPlan& p, int Cout) {
  if (few_takes(p, Cout)) return false;
  if (p.splits > 1) return true;
  switch (p.tile) {
    case 0: return can_pool<TileW32, false, float>();
    case 1: return can_pool<TileW16, false, float>();
    case 2: return can_pool<TileW8, false, float>();
    case 5: return can_pool<TileW32c4, false, float>();
    case 9: return can_pool<TileW32L, false, float>();
    case 10: return can_pool<TileW16L, false, float>();
    case 11: return can_pool<TileW8L, false, float>();
    case 12: return can_pool<TileW8K2, false, float>();
    default: return false;
  }
}

template <bool DGRAD, class E>
static void few_launch(const IgemmPlan& p, const ConvArgs& a, bool pack, hipStream_t st) {
  if (pack)
    filter_pack<DGRAD, FewTile::CK, FewTile::BN, E><<<p.co_tiles * p.nchunks, 256, 0, st>>>(
        (const E*)a.wt, (E*)a.wpk, a.Cin, a.Cout);
  ConvArgs k = a;
  k.tiles_w = cdiv(a.W, FewTile::TW);
  k.tiles_h = cdiv(a.H, FewTile::TH);
  const unsigned grid = (unsigned)(k.tiles_w * k.tiles_h * a.N);
  switch (a.Cout) {
    case 1: conv3x3_few_f32<1, E><<<grid, FewTile::THREADS, 0, st>>>(k); break;
    case 2: conv3x3_few_f32<2, E><<<grid, FewTile::THREADS, 0, st>>>(k); break;
    case 3: conv3x3_few_f32<3, E><<<grid, FewTile::THREADS, 0, st>>>(k); break;
    default: conv3x3_few_f32<4, E><<<grid, FewTile::THREADS, 0, st>>>(k); break;
  }
}

template <bool DGRAD, class E>
static void igemm_dispatch(const IgemmPlan& p, const ConvArgs& a, bool pack, hipStream_t st) {
  if (few_takes(p, a.Cout)) {
    few_launch<DGRAD, E>(p, a, pack, st);
    return;
  }
  switch (p.tile) {
    case 0: igemm_launch<TileW32, DGRAD, false, E>(p, a, pack, st); break;
    case 1: igemm_launch<TileW16, DGRAD, false, E>(p, a, pack, st); break;
    case 2: igemm_launch<TileW8, DGRAD, false, E>(p, a, pack, st); break;
    case 3: igemm_launch<TileW4, DGRAD, false, E>(p, a, pack, st); break;
    case 4: igemm_launch<TileW2, DGRAD, false, E>(p, a, pack, st); break;
    case 5: igemm_launch<TileW32c4, DGRAD, false, E>(p, a, pack, st); break;
    case 6: igemm_launch<TileW32n16, DGRAD, false, E>(p, a, pack, st); break;
    case 7: igemm_launch<Small2, DGRAD, true, E>(p, a, pack, st); break;
    case 8: igemm_launch<Small4, DGRAD, true, E>(p, a, pack, st); break;
    case 9: igemm_launch<TileW32L, DGRAD, false, E>(p, a, pack, st); break;
    case 10: igemm_launch<TileW16L, DGRAD, false, E>(p, a, pack, st); break;
    case 11: igemm_launch<TileW8L, DGRAD, false, E>(p, a, pack, st); break;
    case 12: igemm_launch<TileW8K2, DGRAD, false, E>(p, a, pack, st); break;
    case 13: igemm_launch<Small2K2, DGRAD, true, E>(p, a, pack, st); break;
    default: igemm_launch<Small4K2, DGRAD, true, E>(p, a, pack, st); break;
  }
}

// Packs the filters of a layer for the fp32-MFMA kernels: [tap][ci][co]
// slices of CK input x BN output channels, as the plan's tile stages them
// (CK = 8, BN = 64 but for the 4-channel-chunk and 16-channel-output tiles).
template <bool DGRAD, class E>
static void igemm_pack(const IgemmPlan& p, const void* wt, void* packed, int Cin, int Cout,
                       hipStream_t st) {
  const unsigned g = p.co_tiles * p.nchunks;
  if (p.tile == 5)
    filter_pack<DGRAD, 4, 64, E><<<g, 256, 0, st>>>((const E*)wt, (E*)packed, Cin, Cout);
  else if (p.tile == 6)
    filter_pack<DGRAD, 8, 16, E><<<g, 256, 0, st>>>((const E*)wt, (E*)packed, Cin, Cout);
  else
    filter_pack<DGRAD, 8, 64, E><<<g, 256, 0, st>>>((const E*)wt, (E*)packed, Cin, Cout);
}

}  // namespace sb

// Entry points used by api.hip.
namespace sbh {

// The bf16 MFMA path (conv_bf16.hip) for the bf16 shapes it takes.
size_t conv_bf16_ws(int N, int Cin, int H, int W, int Cout, bool prepacked);
bool conv_bf16_takes(int N, int Cin, int H, int W, int Cout);
int conv_bf16_describe(bool dgrad, int N, int Cin, int H, int W, int Cout, char* buf, size_t len);
size_t conv_bf16_pack_bytes(int N, int Cin, int H, int W, int Cout);
void conv_bf16_pack(bool dgrad, int N, int Cin, int H, int W, int Cout, const void* wt,
                    void* packed, hipStream_t st);
sb_status conv_bf16(bool dgrad, int N, int Cin, int H, int W, int Cout, const void* in,
                    const void* wt, const float* bias, const void* mask, void* out, void* ws,
                    size_t ws_bytes, int relu, bool prepacked, hipStream_t st);

// Workspace of a forward / data-gradient call; prepacked: the filters come
// packed, the workspace holds only the split partials.
size_t conv_igemm_ws(int dtype, int N, int Cin, int H, int W, int Cout, bool prepacked) {
  if (dtype == SB_BF16 && conv_bf16_takes(N, Cin, H, W, Cout))
    return conv_bf16_ws(N, Cin, H, W, Cout, prepacked);
  const int es = (int)dsize(dtype);
  const sb::IgemmPlan p = sb::igemm_plan(N, Cin, H, W, Cout, es, true);
  const sb::IgemmPlan q = sb::igemm_plan(N, Cin, H, W, Cout, es, false);
  if (prepacked) return std::max(p.ws_bytes - p.part_off, q.ws_bytes - q.part_off);
  return std::max(p.ws_bytes, q.ws_bytes);
}

// Bytes of the packed filters.  The packed layout depends on the shape only
// (the whole-image tiles that aligned tensors may take stage the same slices
// as the tiles they replace).
size_t conv_igemm_pack_bytes(int dtype, int N, int Cin, int H, int W, int Cout) {
  if (dtype == SB_BF16 && conv_bf16_takes(N, Cin, H, W, Cout))
    return conv_bf16_pack_bytes(N, Cin, H, W, Cout);
  return sb::igemm_plan(N, Cin, H, W, Cout, (int)dsize(dtype), false).pack_bytes;
}

void conv_bf16_pack_geom(int N, int Cin, int H, int W, int Cout, int* ck, int* bn, int* slices);

// One packing task: the kernel kind (slice geometry and layout) and the
// number of slices of a forward or data-gradient packing.
int conv_igemm_pack_task(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout,
                         const void* wt, void* packed, sb::PackTask* t) {
  int ck, bn, slices, layout;
  if (dtype == SB_BF16 && conv_bf16_takes(N, Cin, H, W, Cout)) {
    conv_bf16_pack_geom(N, Cin, H, W, Cout, &ck, &bn, &slices);
    layout = sb::PackCI8;
  } else {
    const sb::IgemmPlan p = sb::igemm_plan(N, Cin, H, W, Cout, (int)dsize(dtype), false);
    ck = p.tile == 5 ? 4 : 8;
    bn = p.tile == 6 ? 16 : 64;
    slices = p.co_tiles * p.nchunks;
    layout = sb::PackCO;
  }
  t->w = wt;
  t->out = packed;
  t->Cin = Cin;
  t->Cout = Cout;
  t->kind = sb::pack_kind(dgrad, layout, ck, bn);
  return slices;
}

void conv_pack_many(int dtype, const sb::PackBatch& b, hipStream_t st) {
  const unsigned blocks = (unsigned)b.block0[b.ntasks];
  if (dtype == SB_BF16) sb::filter_pack_many<sb::u16><<<blocks, 256, 0, st>>>(b);
  else sb::filter_pack_many<float><<<blocks, 256, 0, st>>>(b);
}

void conv_igemm_pack(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout,
                     const void* wt, void* packed, hipStream_t st) {
  if (dtype == SB_BF16 && conv_bf16_takes(N, Cin, H, W, Cout)) {
    conv_bf16_pack(dgrad, N, Cin, H, W, Cout, wt, packed, st);
    return;
  }
  const sb::IgemmPlan p = sb::igemm_plan(N, Cin, H, W, Cout, (int)dsize(dtype), false);
  if (dtype == SB_BF16) {
    if (dgrad) sb::igemm_pack<true, sb::u16>(p, wt, packed, Cin, Cout, st);
    else sb::igemm_pack<false, sb::u16>(p, wt, packed, Cin, Cout, st);
  } else {
    if (dgrad) sb::igemm_pack<true, float>(p, wt, packed, Cin, Cout, st);
    else sb::igemm_pack<false, float>(p, wt, packed, Cin, Cout, st);
  }
}

// Whether sb_conv3x3_fwd_pool takes an NCHW forward of this shape: fp32,
// even image sizes, and a plan that pools for aligned and unaligned tensors.
bool conv_igemm_pools(int dtype, int N, int Cin, int H, int W, int Cout) {
  if (dtype != SB_F32 || H % 2 || W % 2) return false;
  for (bool aligned : {true, false})
    if (!sb::igemm_pools(sb::igemm_plan(N, Cin, H, W, Cout, 4, aligned), Cout)) return false;
  return true;
}

int conv_igemm_describe(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout,
                        char* buf, size_t len, bool pool) {
  if (dtype == SB_BF16 && conv_bf16_takes(N, Cin, H, W, Cout))
    return conv_bf16_describe(dgrad, N, Cin, H, W, Cout, buf, len);
  sb::IgemmPlan p = sb::igemm_plan(N, Cin, H, W, Cout, (int)dsize(dtype));
  const char* et = dtype == SB_BF16 ? "unsigned short" : "float";
  if (sb::few_takes(p, Cout))
    return snprintf(buf, len, "sb::conv3x3_few_f32<%d, %s> grid=%dx1x1", Cout, et,
                    sb::cdiv(W, sb::FewTile::TW) * sb::cdiv(H, sb::FewTile::TH) * N);
  char name[160];
  snprintf(name, sizeof(name), sb::kTileNames[p.tile], dgrad ? "true" : "false", et);
  if (pool && p.splits == 1) {
    // The pooled instantiation: conv3x3_igemm_f32<T, false, float, WHOLE_H, true>.
    const size_t l = strlen(name);
    if (l > 0 && name[l - 1] == '>')
      snprintf(name + l - 1, sizeof(name) - (l - 1), ", %s, true>",
               H == 8 && (p.tile == 2 || p.tile == 11 || p.tile == 12) ? "true" : "false");
  }
  return snprintf(buf, len, "%s grid=%dx%dx%d", name, p.grid_x, p.co_tiles, p.splits);
}

sb_status conv_igemm(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout,
                     const void* in, const void* wt, const float* bias, const void* mask,
                     void* out, void* ws, size_t ws_bytes, int relu, bool prepacked,
                     hipStream_t st, uint8_t* pool_idx) {
  if (dtype == SB_BF16 && conv_bf16_takes(N, Cin, H, W, Cout))
    return conv_bf16(dgrad, N, Cin, H, W, Cout, in, wt, bias, mask, out, ws, ws_bytes, relu,
                     prepacked, st);
  // The whole-image kernels move 4 elements at a time (16 bytes in fp32, 8 in
  // bf16); the plan only picks them for tensors aligned that far.
  const uintptr_t amask = dtype == SB_BF16 ? 7 : 15;
  const bool aligned = (((uintptr_t)in | (uintptr_t)out | (uintptr_t)mask) & amask) == 0;
  const int64_t es = dsize(dtype);
  sb::IgemmPlan p = sb::igemm_plan(N, Cin, H, W, Cout, (int)es, aligned);
  // Buffer ranges: one block's images of the input, and one output-channel
  // tile's packed filters.
  if ((int64_t)std::min(p.imgs, N) * Cin * H * W * es >= (1ll << 31) ||
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
  if (pool_idx) {
    // Pooled forward: the caller checked conv_igemm_pools (fp32, unsplit,
    // a staged tile); ReLU comes with the pooling.
    if (dgrad || relu || !sb::igemm_pools(p, Cout)) return SB_ERR_UNSUPPORTED;
    a.pool_idx = pool_idx;
  }
  if (dtype == SB_BF16) {
    if (dgrad) sb::igemm_dispatch<true, sb::u16>(p, a, !prepacked, st);
    else sb::igemm_dispatch<false, sb::u16>(p, a, !prepacked, st);
  } else {
    if (dgrad) sb::igemm_dispatch<true, float>(p, a, !prepacked, st);
    else sb::igemm_dispatch<false, float>(p, a, !prepacked, st);
  }
  return launch_status();
}

}  // namespace sbh
