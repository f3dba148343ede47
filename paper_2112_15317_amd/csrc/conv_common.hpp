// conv_common.hpp -- pieces shared by the 3x3 convolution kernels (fp32
// MFMA path and bf16 MFMA path): launch arguments, epilogue, buffer
// resources and the split reduction.
#pragma once

#include "sb_internal.hpp"

#include <type_traits>

namespace sb {

// Element type E of in / wt / mask / out: float or bf16 bits (u16).
// Accumulation, bias and split partials are fp32.
struct ConvArgs {
  const void* in;        // [N][Cin][H][W]
  const void* wt;        // forward filters [K][C][3][3]
  const void* wpk;       // the same, packed by filter_pack (workspace)
  const float* bias;     // [Cout] or null (forward)
  const void* mask;      // [N][Cout][H][W] or null (data gradient)
  void* out;             // [N][Cout][H][W]
  float* part;           // split partials [splits][N][Cout][H][W]
  uint8_t* pool_idx;     // fused ReLU + 2x2 pooling (channel-blocked forward): codes
  int N, Cin, H, W, Cout;
  int tiles_w, tiles_h, nchunks, chunks_per_split, splits, relu;
};

template <class E>
__device__ __forceinline__ float conv_epilogue(const ConvArgs& a, float v, int co, size_t off) {
  if (a.bias) v += a.bias[co];
  if (a.relu && !(v > 0.f)) v = 0.f;
  if (a.mask && !(Elem<E>::load((const E*)a.mask, off) > 0.f)) v = 0.f;
  return v;
}

// Filters are repacked before the convolution (filter_pack) into the order
// the kernels stage them: for output-channel tile t (BN channels) and input-
// channel chunk k (CK channels), 9*CK*BN contiguous elements ordered
// [tap][ci][co], zero where a channel lies past the end.  For the data
// gradient the same pass transposes (co <-> ci) and rotates the taps by 180
// degrees.  A chunk's slice is then one coalesced read, and its LDS rows
// r = tap*CK + ci (stride BN_P) are written by consecutive lanes along a row:
// conflict-free, like the MFMA operand reads (rows r..r+3, 16 consecutive co
// per row, BN_P = 16 mod 64).  The packed filters live in the workspace.
//
// One block per slice: it reads the slice in the filters' own order (runs
// of CK*9 contiguous elements per output channel, or BN*9 per input channel
// for the data gradient), permutes it in LDS and writes it out contiguously.
//
// PackCI8 packs each slice [tap][ci / 8][co][ci % 8] instead: planes of 8
// consecutive input channels per output channel, the operand order of the
// bf16 kernels, whose lanes read 8 consecutive channels (16 bytes).
constexpr int PackCO = 0, PackCI8 = 1;

// Packs slice `slice` of one layer's filters, permuting through `slice_lds`
// (at least slice_lds_bytes<CK, BN, E, LAYOUT>() bytes).
template <int CK, int BN, class E, int LAYOUT>
__host__ __device__ constexpr int slice_lds_elems() {
  return 9 * CK * BN / (LAYOUT == PackCI8 ? 8 : BN) * ((LAYOUT == PackCI8 ? 8 : BN) + 1);
}
template <bool DGRAD, int CK, int BN, class E, int LAYOUT>
__device__ __forceinline__ void pack_slice(const E* __restrict__ w, E* __restrict__ out, int Cin,
                                           int Cout, int slice, E* slice_lds) {
  // Cin, Cout: this convolution's input and output channels (for the data
  // gradient: the forward layer's output and input channels).
  constexpr int SL = 9 * CK * BN;
  constexpr bool CI8 = LAYOUT == PackCI8;
  static_assert(!CI8 || CK % 8 == 0, "whole 8-channel planes");
  // Padded LDS rows (one extra element) keep the permuting writes spread
  // over the banks.
  constexpr int ROW = CI8 ? 8 : BN, RS = ROW + 1;
  constexpr int PT = (SL + 255) / 256;
  const int nchunks = cdiv(Cin, CK);
  const int ct = slice / nchunks, kc = slice - ct * nchunks;   // co tile, chunk
  // Filters whose channel counts are multiples of VEC = 16 / sizeof(E)
  // (4 fp32 or 8 bf16 elements) and 16-byte aligned: every run of
  // consecutive source elements (CK * 9 per output channel, or BN * 9 per
  // input channel for the data gradient) then starts 16-byte aligned and is
  // a multiple of VEC long, so the slice is read in groups of VEC
  // consecutive slice elements with one 16-byte load each.  A group lies in
  // one run; it is read whole when all its elements are in range, element by
  // element otherwise.  The permuted slice goes out in 16-byte pieces too
  // when LDS rows hold whole groups.
  constexpr int VEC = 16 / (int)sizeof(E);
  struct alignas(16) Piece { E e[VEC]; };
  if constexpr (SL % VEC == 0 && (CK * 9) % VEC == 0 && (BN * 9) % VEC == 0) {
    if (Cin % VEC == 0 && Cout % VEC == 0 && ((uintptr_t)w & 15) == 0) {
      constexpr int PTV = (SL / VEC + 255) / 256;
      // Slice element g -> (channel within the run's tile, its source offset).
      auto locate = [&](int g, int& tap, int& cc, int& nn, size_t& src) {
        if (!DGRAD) {                                 // g = (nn, cc, tap), tap fastest
          nn = g / (CK * 9);
          const int r = g - nn * (CK * 9);
          cc = r / 9;
          tap = r - cc * 9;
          src = ((size_t)(ct * BN + nn) * Cin + kc * CK + cc) * 9 + tap;
        } else {                                      // g = (cc, nn, t), t fastest
          cc = g / (BN * 9);
          const int r = g - cc * (BN * 9);
          nn = r / 9;
          const int t = r - nn * 9;
          tap = 8 - t;
          src = ((size_t)(kc * CK + cc) * Cout + ct * BN + nn) * 9 + t;
        }
      };
      auto live = [&](int cc, int nn) { return ct * BN + nn < Cout && kc * CK + cc < Cin; };
      Piece v[PTV];
#pragma unroll
      for (int i = 0; i < PTV; ++i) {
        const int g = (threadIdx.x + i * 256) * VEC;
        if (g >= SL) continue;
        int tap, cc, nn, tapl, ccl, nnl;
        size_t src, srcl;
        locate(g, tap, cc, nn, src);
        locate(g + VEC - 1, tapl, ccl, nnl, srcl);
        if (live(cc, nn) && live(ccl, nnl)) {         // the group's first and last in range
          v[i] = *reinterpret_cast<const Piece*>(w + src);
        } else {
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            int te, ce, ne;
            size_t se;
            locate(g + e, te, ce, ne, se);
            v[i].e[e] = live(ce, ne) ? w[se] : E{};
          }
        }
      }
#pragma unroll
      for (int i = 0; i < PTV; ++i) {
        const int g0 = (threadIdx.x + i * 256) * VEC;
        if (g0 >= SL) continue;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          int tap, cc, nn;
          size_t src;
          locate(g0 + e, tap, cc, nn, src);
          slice_lds[CI8 ? ((tap * (CK / 8) + cc / 8) * BN + nn) * RS + cc % 8
                        : (tap * CK + cc) * RS + nn] = v[i].e[e];
        }
      }
      __syncthreads();
      E* dst = out + (size_t)slice * SL;
      if (ROW % VEC == 0 && ((uintptr_t)out & 15) == 0) {
        // A group of VEC never crosses an LDS row, and each slice starts
        // 16-byte aligned (SL % VEC == 0).
        for (int e = threadIdx.x * VEC; e < SL; e += 256 * VEC) {
          const E* l = slice_lds + (e / ROW) * RS + e % ROW;
          Piece q;
#pragma unroll
          for (int k = 0; k < VEC; ++k) q.e[k] = l[k];
          *reinterpret_cast<Piece*>(dst + e) = q;
        }
      } else {
        for (int e = threadIdx.x; e < SL; e += 256) dst[e] = slice_lds[(e / ROW) * RS + e % ROW];
      }
      return;
    }
  }
  // All loads first (PT per thread in flight), then the LDS permutation.
  E v[PT];
  int pos[PT];
#pragma unroll
  for (int i = 0; i < PT; ++i) {
    const int g = threadIdx.x + i * 256;
    int tap, cc, nn;
    size_t src;
    if (!DGRAD) {                                     // g = (nn, cc, tap), tap fastest
      nn = g / (CK * 9);
      const int r = g - nn * (CK * 9);
      cc = r / 9;
      tap = r - cc * 9;
      src = ((size_t)(ct * BN + nn) * Cin + kc * CK + cc) * 9 + tap;
    } else {                                          // g = (cc, nn, t), t fastest
      cc = g / (BN * 9);
      const int r = g - cc * (BN * 9);
      nn = r / 9;
      const int t = r - nn * 9;
      tap = 8 - t;
      src = ((size_t)(kc * CK + cc) * Cout + ct * BN + nn) * 9 + t;
    }
    const bool ok = g < SL && ct * BN + nn < Cout && kc * CK + cc < Cin;
    v[i] = ok ? w[src] : E{};
    pos[i] = g < SL ? (CI8 ? ((tap * (CK / 8) + cc / 8) * BN + nn) * RS + cc % 8
                           : (tap * CK + cc) * RS + nn)
                    : -1;
  }
#pragma unroll
  for (int i = 0; i < PT; ++i)
    if (pos[i] >= 0) slice_lds[pos[i]] = v[i];
  __syncthreads();
  E* dst = out + (size_t)slice * SL;
  for (int e = threadIdx.x; e < SL; e += 256) dst[e] = slice_lds[(e / ROW) * RS + e % ROW];
}

// One block per slice of one layer.
template <bool DGRAD, int CK, int BN, class E, int LAYOUT = PackCO>
__global__ __launch_bounds__(256) void filter_pack(const E* __restrict__ w, E* __restrict__ out,
                                                   int Cin, int Cout) {
  __shared__ E slice_lds[slice_lds_elems<CK, BN, E, LAYOUT>()];
  pack_slice<DGRAD, CK, BN, E, LAYOUT>(w, out, Cin, Cout, blockIdx.x, slice_lds);
}

// Several layers' (and passes') filters in one launch: a pack task per
// (filters, pass); the blocks of task t are block0[t] .. block0[t+1]-1, one
// per slice.  `kind` names the slice geometry (pack_kind()).  One launch
// instead of one per task: a pack moves little data, so each separate
// launch would cost mostly its own ramp-up and drain.
constexpr int kMaxPackTasks = 64;
struct PackTask {
  const void* w;
  void* out;
  int Cin, Cout;   // of the convolution (for the data gradient, the transposed one)
  int kind;
};
struct PackBatch {
  PackTask t[kMaxPackTasks];
  int block0[kMaxPackTasks + 1];
  int ntasks;
};
// kind = DGRAD | CI8 << 1 | ck_code << 2 | bn_code << 4, with ck_code 0, 1, 2
// for CK = 4, 8, 16 and bn_code 0, 1, 2 for BN = 16, 32, 64.
__host__ __device__ constexpr int pack_kind(bool dgrad, int layout, int ck, int bn) {
  return (dgrad ? 1 : 0) | (layout == PackCI8 ? 2 : 0) | ((ck == 4 ? 0 : ck == 8 ? 1 : 2) << 2) |
         ((bn == 16 ? 0 : bn == 32 ? 1 : 2) << 4);
}

// fp32 filters only take the PackCO kinds (the bf16 kernels' PackCI8 slices
// are bf16), so the fp32 kernel sizes its LDS for those alone: the larger
// PackCI8 buffer would cut the resident blocks per CU by more than half.
template <class E>
__global__ __launch_bounds__(256) void filter_pack_many(PackBatch b) {
  constexpr bool F32 = std::is_same<E, float>::value;
  constexpr int LDS = !F32 && slice_lds_elems<16, 64, E, PackCI8>() >
                                  slice_lds_elems<8, 64, E, PackCO>()
                          ? slice_lds_elems<16, 64, E, PackCI8>()
                          : slice_lds_elems<8, 64, E, PackCO>();
  __shared__ E slice_lds[LDS];
  const int blk = blockIdx.x;
  int t = 0;
  while (t + 1 < b.ntasks && b.block0[t + 1] <= blk) ++t;
  const PackTask& k = b.t[t];
  const int slice = blk - b.block0[t];
  const E* w = (const E*)k.w;
  E* out = (E*)k.out;
#define SB_PACK_CASE(DG, LAY, CK, BN)                                                      \
  case pack_kind(DG, LAY, CK, BN):                                                         \
    pack_slice<DG, CK, BN, E, LAY>(w, out, k.Cin, k.Cout, slice, slice_lds);                \
    break;
  switch (k.kind) {
    SB_PACK_CASE(false, PackCO, 8, 64)
    SB_PACK_CASE(true, PackCO, 8, 64)
    SB_PACK_CASE(false, PackCO, 4, 64)
    SB_PACK_CASE(true, PackCO, 4, 64)
    SB_PACK_CASE(false, PackCO, 8, 16)
    SB_PACK_CASE(true, PackCO, 8, 16)
    default:
      if constexpr (!F32) {
        switch (k.kind) {
          SB_PACK_CASE(false, PackCI8, 16, 64)
          SB_PACK_CASE(true, PackCI8, 16, 64)
          SB_PACK_CASE(false, PackCI8, 16, 32)
          SB_PACK_CASE(true, PackCI8, 16, 32)
          default: break;
        }
      }
      break;
  }
#undef SB_PACK_CASE
}

// Buffer resources of a block: its images of the input (from image n0 on)
// and the whole filter tensor.
template <class E>
__device__ __forceinline__ rsrc_t input_rsrc(const ConvArgs& a, int n0, int imgs) {
  const size_t img = (size_t)a.Cin * a.H * a.W;
  const int cnt = min(imgs, a.N - n0);
  return make_rsrc((const E*)a.in + n0 * img, (uint32_t)(cnt * img * sizeof(E)));
}
// The packed filter slices of output-channel tile `ct` (all chunks).
template <class E, int WTS>
__device__ __forceinline__ rsrc_t packed_rsrc(const ConvArgs& a, int ct) {
  return make_rsrc((const E*)a.wpk + (size_t)ct * a.nchunks * WTS,
                   (uint32_t)((size_t)a.nchunks * WTS * sizeof(E)));
}

// Channel of flat output element i: NCHW, or channel-blocked (C8: blocks
// of 8 channels innermost per pixel).
template <bool C8>
__device__ __forceinline__ int flat_channel(size_t i, int Cout, int HWs) {
  if (C8) return (int)(((i >> 3) / HWs) % (size_t)(Cout >> 3)) * 8 + (int)(i & 7);
  return (int)((i / HWs) % Cout);
}
// Sum of the split partials in a fixed order, then the epilogue.
template <class E, bool C8 = false>
__global__ __launch_bounds__(256) void conv_splitk_reduce(
    const float* __restrict__ part, int splits, size_t total, int Cout, int HWs,
    const float* __restrict__ bias, int relu, const E* __restrict__ mask,
    E* __restrict__ out) {
  __shared__ float lds[256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t i = (size_t)blockIdx.x * 64 + lane;
  float v = SplitSum{part, splits, total, total}(i, wave, lds, lane);
  if (wave != 0 || i >= total) return;
  if (bias) v += bias[flat_channel<C8>(i, Cout, HWs)];
  if (relu && !(v > 0.f)) v = 0.f;
  if (mask && !(Elem<E>::load(mask, i) > 0.f)) v = 0.f;
  Elem<E>::store(out, i, v);
}

// The same for 4 consecutive outputs per thread (total a multiple of 4 and
// the partials 16-byte aligned): 16-byte partial loads, all splits of a
// thread's outputs summed in one thread in split order.
template <class E, bool C8 = false>
__global__ __launch_bounds__(256) void conv_splitk_reduce4(
    const float* __restrict__ part, int splits, size_t total, int Cout, int HWs,
    const float* __restrict__ bias, int relu, const E* __restrict__ mask,
    E* __restrict__ out) {
  const size_t i4 = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i4 >= total) return;
  f4 v = split_sum4(part, splits, total, i4);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const size_t i = i4 + j;
    float r = v[j];
    if (bias) r += bias[flat_channel<C8>(i, Cout, HWs)];
    if (relu && !(r > 0.f)) r = 0.f;
    if (mask && !(Elem<E>::load(mask, i) > 0.f)) r = 0.f;
    Elem<E>::store(out, i, r);
  }
}

// Split reduction of a forward pooled in the same call (NCHW, even H and
// W): per pooled output, the window's four sums over the splits in
// increasing order (conv_splitk_reduce4's order) plus the bias, then ReLU
// and 2x2 max pooling as relu_maxpool_fwd takes them: the first maximum in
// row-major window order (strict >), the maximum if positive, else +0, and
// bit 7 of the code for the latter.
template <class E, bool VEC>
__global__ __launch_bounds__(256) void conv_splitk_reduce_pool(
    const float* __restrict__ part, int splits, size_t total, int Cout, int H, int W,
    const float* __restrict__ bias, E* __restrict__ out, uint8_t* __restrict__ idx) {
  const int Hh = H / 2, Wh = W / 2;
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= total / 4) return;
  const int ow = (int)(q % Wh);
  const size_t r = q / Wh;
  const int oh = (int)(r % Hh);
  const size_t nc = r / Hh;                               // n * Cout + co
  // The window's two rows are pairs of adjacent floats (W and the window's
  // first column even), read as 8-byte pieces when the partials are 8-byte
  // aligned (VEC).
  const size_t p0 = (nc * H + 2 * oh) * W + 2 * ow;
  const float bv = bias ? bias[nc % Cout] : 0.f;
  typedef float f2 __attribute__((ext_vector_type(2)));
  f2 top = {0.f, 0.f}, bot = {0.f, 0.f};
  for (int sp = 0; sp < splits; ++sp) {
    const float* ps = part + (size_t)sp * total;
    if (VEC) {
      top += *reinterpret_cast<const f2*>(ps + p0);
      bot += *reinterpret_cast<const f2*>(ps + p0 + W);
    } else {
      top += f2{ps[p0], ps[p0 + 1]};
      bot += f2{ps[p0 + W], ps[p0 + W + 1]};
    }
  }
  const float v[4] = {top[0] + bv, top[1] + bv, bot[0] + bv, bot[1] + bv};
  float m = v[0];
  uint32_t c = 0;
#pragma unroll
  for (int k = 1; k < 4; ++k)
    if (v[k] > m) { m = v[k]; c = (uint32_t)k; }
  const bool pos = m > 0.f;
  Elem<E>::store(out, q, pos ? m : 0.f);
  idx[q] = (uint8_t)(c | (pos ? 0u : 0x80u));
}

// Launches the split reduction of a convolution pass: the 4-wide form when
// the sizes allow, else one output per lane.
template <class E, bool C8 = false>
inline void launch_splitk_reduce(const float* part, int splits, size_t total, int Cout, int HWs,
                                 const float* bias, int relu, const E* mask, E* out,
                                 hipStream_t st) {
  if (total % 4 == 0 && ((uintptr_t)part & 15) == 0)
    conv_splitk_reduce4<E, C8><<<(unsigned)((total / 4 + 255) / 256), 256, 0, st>>>(
        part, splits, total, Cout, HWs, bias, relu, mask, out);
  else
    conv_splitk_reduce<E, C8><<<(unsigned)((total + 63) / 64), 256, 0, st>>>(
        part, splits, total, Cout, HWs, bias, relu, mask, out);
}

}  // namespace sb
