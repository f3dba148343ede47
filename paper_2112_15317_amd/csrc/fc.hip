// fc.hip -- FC column shard forward and backward (sec. 3.1: a LINEAR layer
// split to 1/K of its outputs, run on the batch the modulo layer gathers;
// its backward yields this shard's partial gradient over the full input).
//
//   forward   Y   = X * W_sh (+ b) (ReLU)       [m x ns] = [m x kin][kin x ns]
//   backward  dXp = G * W_sh^T                  [m x kin]
//             dW  = (dW +) X^T * G              [kin x ns]
//             db  = (db +) column sums of G     [ns]
// with G = dY, or dY * [mask > 0] (ReLU of this shard's output).
//
// SB_BF16: x, w_shard, y, dy, the ReLU mask and dx_partial are bfloat16;
// the kernel widens them exactly to fp32 as it stages them (so the products
// and sums are the fp32 path's, on the same fp32 MFMA) and rounds y and
// dx_partial to nearest-even on store; dW and db stay fp32.
//
// One fp32 MFMA GEMM kernel (gemm_f32 below) serves the three products;
// the backward's bias gradient is added up inside the dW product.  Tile
// shapes and reduction splits are chosen per shape (gemm_plan).
#include "sb_internal.hpp"

#include <algorithm>
#include <type_traits>
#include <mutex>

namespace sb {

// ---------------------------------------------------------------------------
// GEMM core.  C = epi(A * B) with A [M x K], B [K x N], fp32 accumulation on
// v_mfma_f32_32x32x2_f32 (one 32x32 output block per instruction).  Block
// tile BM x BN x 32 (BM, BN in {64, 128}), four waves in a 2 x 2 layout, each
// owning (BM/2) x (BN/2) as (BM/64) x (BN/64) MFMA blocks.
//
// MFMA lane layout (32x32x2, fp32): lane l supplies A[l % 32][k_h] and
// B[k_h][l % 32] with k_h the half-wave's k (h = l / 32); it receives
// D[8 (r / 4) + 4 h + r % 4][l % 32] in accumulator element r.
//
// The reduction runs in chunks of 8 k; MFMA step j (0..3) of a chunk takes
// k = 4 h + j from half-wave h, for both operands (any fixed pairing of the
// reduction index gives the same sum up to rounding).  Each operand keeps
// the layout it has in memory when it is staged in LDS:
//   * contiguous along k ("K-contiguous"): [row][k], row stride 36 floats;
//     a lane reads its 4 k of a chunk as one 16-byte read (16-byte units
//     9 * row + h: the 16 lanes of a read phase hit distinct banks);
//   * contiguous along its row index: [k][row], k stride BM + 8 floats; a
//     lane reads one float per step (the two half-waves read rows 4 k apart,
//     4 (BM + 8) = 32 mod 64 banks: all 64 lanes on distinct banks).
// Global loads are raw buffer loads whose out-of-range offsets read 0, so
// ragged edges need no branches around the loads; the ReLU mask of dY is
// applied when the operand is stored to LDS.  Operands of type E (fp32, or
// bf16 bits widened exactly) are staged as fp32.
//
// A long reduction over few output tiles is split over `splits` ranges of
// k; each split writes fp32 partials [split][M][N] and gemm_splitk_epilogue
// sums them in a fixed order.  Blocks are numbered split-major and dealt to
// the 8 XCDs in contiguous ranges of that order, so the blocks one XCD runs
// share operand slices in its L2 (with 8 splits: one split per XCD).
//
// colsum (the FC bias gradient): blocks of the first row tile also add up,
// on the vector ALU beside the MFMAs, the B values they feed their MFMAs;
// the two half-waves' sums are combined and the waves of the first row of
// waves (the other row reads the same B) write the column sums.
constexpr int GBK = 32;
constexpr int RK = GBK + 4;                          // [row][k] row stride (floats)

template <int R> struct OpGeom {
  static constexpr int RR = R + 8;                   // [k][row] k stride (floats)
  static constexpr int KC_FLOATS = R * RK;
  static constexpr int RC_FLOATS = GBK * RR;
  static constexpr int GROUPS = R * GBK / 4 / 256;   // 4-element groups per thread
};

template <int BM, int BN>
struct GemmTile {
  static constexpr int OPA = OpGeom<BM>::KC_FLOATS > OpGeom<BM>::RC_FLOATS
                                 ? OpGeom<BM>::KC_FLOATS : OpGeom<BM>::RC_FLOATS;
  static constexpr int OPB = OpGeom<BN>::KC_FLOATS > OpGeom<BN>::RC_FLOATS
                                 ? OpGeom<BN>::KC_FLOATS : OpGeom<BN>::RC_FLOATS;
  static constexpr int BUF = OPA + OPB;
  static constexpr size_t LDS_BYTES = 2 * BUF * sizeof(float);
  static constexpr int RB = BM / 64, CB = BN / 64;   // MFMA blocks per wave
  static_assert(LDS_BYTES <= 80 * 1024, "two blocks per CU");
};

struct GemmArgs {
  const void* a; int lda;              // A element (m,k): A_KC ? a[m*lda+k] : a[k*lda+m]
  const void* amask;                   // optional mask, same layout/stride as a
  const void* b; int ldb;              // B element (k,n): B_KC ? b[n*ldb+k] : b[k*ldb+n]
  const void* bmask;
  void* c; int ldc;                    // C[m*ldc + n] (type CE), or fp32 partials
  int M, N, K;
  int mt, nt, splits, k_per_split;
  const float* bias; int relu; int accumulate;
  float* colsum; int colsum_acc;       // column sums of B (k < K), or null
};

// One operand's staging: R x 32 elements in groups of 4, OpGeom<R>::GROUPS
// per thread.  K-contiguous: group g = (row g / 8, k quad g % 8), so the 8
// threads of a row read its 128 contiguous bytes of the tile.
// Row-contiguous: group g = (row quad g % (R/4), k g / (R/4)).  A thread's
// groups keep their rows and in-tile k for the whole reduction, so their
// element offsets (at k = 0) and row checks are worked out once; a tile
// adds its first k.  VEC loads a group with one vector load (aligned, whole
// groups in range); otherwise element by element.  The mask (when there is
// one) is applied when the tile is stored to LDS, so no load waits for
// another before the store.
template <int R, bool KC, bool VEC, class E>
struct Stage {
  static constexpr int G = OpGeom<R>::GROUPS;
  f4 v[G], m[G];
  int off0[G], kin[G];       // element offset at k = 0 (-1: row outside); k in the tile
  int ld;
  __device__ __forceinline__ void init(int ld_, int rows, int r0, int tid) {
    ld = ld_;
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const int g = tid + i * 256;
      const int row = KC ? r0 + g / 8 : r0 + (g % (R / 4)) * 4;
      kin[i] = KC ? (g % 8) * 4 : g / (R / 4);
      off0[i] = row < rows ? (KC ? row * ld + kin[i] : kin[i] * ld + row) : -1;
    }
  }
  __device__ __forceinline__ void load(rsrc_t r, rsrc_t rm, bool masked, int rows, int r0,
                                       int k0, int ke, int tid) {
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const int k = k0 + kin[i];
      const int koff = KC ? k0 : k0 * ld;
      if (VEC) {
        const uint32_t off = (off0[i] >= 0 && k < ke)
                                 ? (uint32_t)(off0[i] + koff) * (uint32_t)sizeof(E) : kOOB;
        v[i] = BufLoad<E>::four(r, off);
        if (masked) m[i] = BufLoad<E>::four(rm, off);
      } else {
        const int g = tid + i * 256;
        const int row = KC ? r0 + g / 8 : r0 + (g % (R / 4)) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rr = KC ? row : row + e, kk = KC ? k + e : k;
          const bool ok = rr < rows && kk < ke;
          const uint32_t off =
              ok ? (uint32_t)(KC ? rr * ld + kk : kk * ld + rr) * (uint32_t)sizeof(E) : kOOB;
          v[i][e] = BufLoad<E>::one(r, off);
          if (masked) m[i][e] = BufLoad<E>::one(rm, off);
        }
      }
    }
  }
  __device__ __forceinline__ void store(float* S, bool masked, int tid) const {
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const int g = tid + i * 256;
      float* p = KC ? S + (g / 8) * RK + (g % 8) * 4 : S + (g / (R / 4)) * OpGeom<R>::RR +
                                                         (g % (R / 4)) * 4;
      f4 x = v[i];
      if (masked) {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = m[i][e] > 0.f ? x[e] : 0.f;
      }
      *reinterpret_cast<f4*>(p) = x;
    }
  }
};

// Operand values of chunk c (8 k) for NB 32-row blocks of a wave:
// f[blk][j] = element (row row0 + 32 blk + l % 32, k = 8 c + 4 h + j).
template <int R, bool KC, int NB>
__device__ __forceinline__ void frag32(const float* S, int row0, int c, int h, int l32,
                                       f4 (&f)[NB]) {
#pragma unroll
  for (int blk = 0; blk < NB; ++blk) {
    const int row = row0 + blk * 32 + l32;
    if (KC) {
      f[blk] = *reinterpret_cast<const f4*>(S + row * RK + c * 8 + h * 4);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) f[blk][j] = S[(c * 8 + h * 4 + j) * OpGeom<R>::RR + row];
    }
  }
}

typedef float f16v __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f16v mfma32x32x2(float a, float b, f16v c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// The block's (row tile, column tile, split) from its linear id: dealt to
// the 8 XCDs in contiguous ranges of the split-major order when the grid is
// a multiple of 8 blocks.
__device__ __forceinline__ void gemm_block(const GemmArgs& g, int& mtile, int& ntile, int& split) {
  const int nb = g.mt * g.nt * g.splits;
  int h = blockIdx.x;
  if (nb % 8 == 0) h = (h % 8) * (nb / 8) + h / 8;
  const int tiles = g.mt * g.nt;
  split = h / tiles;
  const int t = h - split * tiles;
  mtile = t / g.nt;
  ntile = t - mtile * g.nt;
}

template <int BM, int BN, bool A_KC, bool B_KC, bool VEC, class E, class CE, bool AMK, bool BMK>
__global__ __launch_bounds__(256, 2) void gemm_f32(GemmArgs g) {
  using T = GemmTile<BM, BN>;
  extern __shared__ float lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int h = lane >> 5, l32 = lane & 31;
  int mtile, ntile, split;
  gemm_block(g, mtile, ntile, split);
  const int m0 = mtile * BM, n0 = ntile * BN;
  const int kb = split * g.k_per_split;
  const int ke = min(g.K, kb + g.k_per_split);
  // Whole operand tensors (the host keeps them below 2^31 bytes).
  const size_t a_elems = A_KC ? (size_t)(g.M - 1) * g.lda + g.K : (size_t)(g.K - 1) * g.lda + g.M;
  const size_t b_elems = B_KC ? (size_t)(g.N - 1) * g.ldb + g.K : (size_t)(g.K - 1) * g.ldb + g.N;
  const rsrc_t ra = make_rsrc(g.a, (uint32_t)(a_elems * sizeof(E)));
  const rsrc_t rb = make_rsrc(g.b, (uint32_t)(b_elems * sizeof(E)));
  const rsrc_t ram = make_rsrc(g.amask ? g.amask : g.a, (uint32_t)(a_elems * sizeof(E)));
  const rsrc_t rbm = make_rsrc(g.bmask ? g.bmask : g.b, (uint32_t)(b_elems * sizeof(E)));
  constexpr bool amasked = AMK, bmasked = BMK;
  const bool do_colsum = g.colsum != nullptr && mtile == 0;

  f16v acc[T::RB][T::CB];
#pragma unroll
  for (int i = 0; i < T::RB; ++i)
#pragma unroll
    for (int j = 0; j < T::CB; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  float csum[T::CB];
#pragma unroll
  for (int j = 0; j < T::CB; ++j) csum[j] = 0.f;

  Stage<BM, A_KC, VEC, E> sa[2];
  Stage<BN, B_KC, VEC, E> sb_[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    sa[q].init(g.lda, g.M, m0, tid);
    sb_[q].init(g.ldb, g.N, n0, tid);
  }
  auto Abuf = [&](int b) { return lds + b * T::BUF; };
  auto Bbuf = [&](int b) { return lds + b * T::BUF + T::OPA; };

  const int nk = ke > kb ? cdiv(ke - kb, GBK) : 0;
  sa[0].load(ra, ram, amasked, g.M, m0, kb, ke, tid);
  sb_[0].load(rb, rbm, bmasked, g.N, n0, kb, ke, tid);
  sa[1].load(ra, ram, amasked, g.M, m0, kb + GBK, ke, tid);
  sb_[1].load(rb, rbm, bmasked, g.N, n0, kb + GBK, ke, tid);
  sa[0].store(Abuf(0), amasked, tid);
  sb_[0].store(Bbuf(0), bmasked, tid);
  sa[0].load(ra, ram, amasked, g.M, m0, kb + 2 * GBK, ke, tid);
  sb_[0].load(rb, rbm, bmasked, g.N, n0, kb + 2 * GBK, ke, tid);
  __syncthreads();
  // Tile j's operands travel in register set j % 2.  Per tile t: the first
  // chunk's operands are read from LDS, tile t + 1 is stored to the other
  // LDS buffer and tile t + 3 is requested into the register set that store
  // frees (two tiles ahead of its own store); then each chunk's MFMAs run
  // while the following chunk's operands are read.
  auto step = [&](auto P, int t) {
    constexpr int Q = decltype(P)::value;          // t % 2
    const int buf = Q;
    const float* A = Abuf(buf);
    const float* B = Bbuf(buf);
    f4 fa[T::RB], fb[T::CB], na[T::RB], nb[T::CB];
    frag32<BM, A_KC, T::RB>(A, wm * (BM / 2), 0, h, l32, fa);
    frag32<BN, B_KC, T::CB>(B, wn * (BN / 2), 0, h, l32, fb);
    // Unconditional: a tile past the end loads as zeros (every offset out
    // of range) and its LDS copy is never read, so the loop body has one
    // path and the compiler counts outstanding loads exactly.
    sa[Q ^ 1].store(Abuf(buf ^ 1), amasked, tid);
    sb_[Q ^ 1].store(Bbuf(buf ^ 1), bmasked, tid);
    sa[Q ^ 1].load(ra, ram, amasked, g.M, m0, kb + (t + 3) * GBK, ke, tid);
    sb_[Q ^ 1].load(rb, rbm, bmasked, g.N, n0, kb + (t + 3) * GBK, ke, tid);
#pragma unroll
    for (int c = 0; c < GBK / 8; ++c) {
      if (c + 1 < GBK / 8) {
        frag32<BM, A_KC, T::RB>(A, wm * (BM / 2), c + 1, h, l32, na);
        frag32<BN, B_KC, T::CB>(B, wn * (BN / 2), c + 1, h, l32, nb);
      }
      // Keep those reads ahead of this chunk's MFMAs (the scheduler would
      // otherwise sink them next to their first use).
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < T::RB; ++i)
#pragma unroll
          for (int n = 0; n < T::CB; ++n) acc[i][n] = mfma32x32x2(fa[i][j], fb[n][j], acc[i][n]);
      if (do_colsum) {
#pragma unroll
        for (int n = 0; n < T::CB; ++n) csum[n] += (fb[n][0] + fb[n][1]) + (fb[n][2] + fb[n][3]);
      }
      if (c + 1 < GBK / 8) {
#pragma unroll
        for (int i = 0; i < T::RB; ++i) fa[i] = na[i];
#pragma unroll
        for (int n = 0; n < T::CB; ++n) fb[n] = nb[n];
      }
    }
    __syncthreads();
  };
  int t = 0;
  for (; t + 1 < nk; t += 2) {
    step(std::integral_constant<int, 0>{}, t);
    step(std::integral_constant<int, 1>{}, t + 1);
  }
  if (t < nk) step(std::integral_constant<int, 0>{}, t);

  if (do_colsum) {
#pragma unroll
    for (int n = 0; n < T::CB; ++n) {
      const float s = csum[n] + __shfl_xor(csum[n], 32, 64);
      const int col = n0 + wn * (BN / 2) + n * 32 + l32;
      if (wm == 0 && h == 0 && col < g.N)
        g.colsum[col] = g.colsum_acc ? g.colsum[col] + s : s;
    }
  }

  // acc[i][n] element r holds C[m0 + wm*BM/2 + 32 i + 8 (r/4) + 4 h + r%4]
  //                            [n0 + wn*BN/2 + 32 n + l32].
  const bool partial = g.splits > 1;
  float* part = partial ? (float*)g.c + (size_t)split * g.M * g.ldc : nullptr;
  CE* dst = (CE*)g.c;
#pragma unroll
  for (int n = 0; n < T::CB; ++n) {
    const int col = n0 + wn * (BN / 2) + n * 32 + l32;
    if (col >= g.N) continue;
    const float bv = (!partial && g.bias) ? g.bias[col] : 0.f;
#pragma unroll
    for (int i = 0; i < T::RB; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * (BM / 2) + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (m >= g.M) continue;
        float v = acc[i][n][r];
        const size_t o = (size_t)m * g.ldc + col;
        if (partial) {
          part[o] = v;
          continue;
        }
        v += bv;
        if (g.relu && !(v > 0.f)) v = 0.f;
        if (g.accumulate) v += Elem<CE>::load(dst, o);
        Elem<CE>::store(dst, o, v);
      }
  }
}

// out[m, n] = epi(sum_s part[s][m][n]): + bias[n], ReLU, + out (accumulate),
// rounded to the output type CE.  Four consecutive outputs per thread when
// N is a multiple of 4 (the splits summed in order for each of them).
template <class CE>
__global__ __launch_bounds__(256) void gemm_splitk_epilogue(
    const float* __restrict__ part, int splits, int M, int N, CE* __restrict__ out, int ldo,
    const float* __restrict__ bias, int relu, int accumulate) {
  const size_t i4 = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i4 >= (size_t)M * N) return;
  const size_t stride = (size_t)M * N;
  if (N % 4 == 0) {
    const f4 v = split_sum4(part, splits, stride, i4);
    const int m = (int)(i4 / N), n = (int)(i4 - (size_t)m * N);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float x = v[e];
      if (bias) x += bias[n + e];
      if (relu && !(x > 0.f)) x = 0.f;
      const size_t o = (size_t)m * ldo + n + e;
      if (accumulate) x += Elem<CE>::load(out, o);
      Elem<CE>::store(out, o, x);
    }
    return;
  }
  for (int e = 0; e < 4; ++e) {
    const size_t i = i4 + e;
    if (i >= (size_t)M * N) return;
    const int m = (int)(i / N), n = (int)(i - (size_t)m * N);
    float x = 0.f;
    for (int s = 0; s < splits; ++s) x += part[(size_t)s * stride + i];
    if (bias) x += bias[n];
    if (relu && !(x > 0.f)) x = 0.f;
    const size_t o = (size_t)m * ldo + n;
    if (accumulate) x += Elem<CE>::load(out, o);
    Elem<CE>::store(out, o, x);
  }
}

// db[j] = (db[j] +) sum_i G[i][j], for the plans whose GEMM cannot add the
// column sums itself (a split reduction).  A block owns 64 columns; its 16
// waves sum every 16th row (four independent partial sums each, combined in
// a fixed order), then the wave sums are added in order through LDS.
template <class E>
__global__ __launch_bounds__(1024) void col_sum(const E* __restrict__ dy,
                                                const E* __restrict__ mask, int M, int N,
                                                int ld, float* __restrict__ db, int accumulate) {
  __shared__ float part[16][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + lane;
  float s4[4] = {0.f, 0.f, 0.f, 0.f};
  if (j < N) {
    int u = 0;
    for (int i = wave; i < M; i += 16, u = (u + 1) & 3) {
      const size_t o = (size_t)i * ld + j;
      float v = Elem<E>::load(dy, o);
      if (mask && !(Elem<E>::load(mask, o) > 0.f)) v = 0.f;
      s4[u] += v;
    }
  }
  part[wave][lane] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
  __syncthreads();
  if (wave != 0 || j >= N) return;
  float v = 0.f;
#pragma unroll
  for (int w = 0; w < 16; ++w) v += part[w][lane];
  db[j] = accumulate ? db[j] + v : v;
}

// Tile shape and split of one GEMM.  Candidates: 128x128, 128x64 and 64x64
// block tiles, 1..16 splits of the reduction (each at least 4 k-tiles).
// Measured on the FC shard's shapes, a block alone on its CU waits on its
// operand loads, while two blocks per CU hide each other's waits, and
// splits cost their partials and a reduction launch.  So the plan takes the
// most blocks up to 512 (two per CU), then the fewest splits, then the
// largest tile.
struct GemmPlan { int bm, bn, mt, nt, splits, kps; size_t ws_bytes; };

static GemmPlan gemm_plan(int M, int N, int K, int /*esize*/) {
  static const int kTiles[3][2] = {{128, 128}, {128, 64}, {64, 64}};
  GemmPlan best{};
  long best_blocks = 0;
  const int ktiles = cdiv(K, GBK);
  for (const auto& t : kTiles) {
    const int mt = cdiv(M, t[0]), nt = cdiv(N, t[1]);
    for (int s = 1; s <= 16; s *= 2) {
      if (s > 1 && ktiles / s < 4) break;
      const int tps = cdiv(ktiles, s);
      const int splits = cdiv(ktiles, tps);
      if (splits != s) continue;
      const long blocks = std::min<long>((long)mt * nt * splits, 512);
      const bool better = best.mt == 0 || blocks > best_blocks ||
                          (blocks == best_blocks && splits < best.splits);
      if (better) {
        best = GemmPlan{t[0], t[1], mt, nt, splits, tps * GBK, 0};
        best_blocks = blocks;
      }
    }
  }
  best.ws_bytes = best.splits > 1 ? (size_t)best.splits * M * N * sizeof(float) : 0;
  return best;
}

// 4-element groups load as one vector (16 bytes fp32, 8 bytes bf16).
template <class E>
static bool vec_ok(const void* p, int ld, int contiguous_extent) {
  return ((uintptr_t)p & (4 * sizeof(E) - 1)) == 0 && ld % 4 == 0 && contiguous_extent % 4 == 0;
}

template <int BM, int BN, bool AK, bool BK, bool VEC, class E, class CE, bool AMK, bool BMK>
static void gemm_launch_t(const GemmPlan& p, const GemmArgs& g, hipStream_t st) {
  using T = GemmTile<BM, BN>;
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute((const void*)gemm_f32<BM, BN, AK, BK, VEC, E, CE, AMK, BMK>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)T::LDS_BYTES);
  });
  gemm_f32<BM, BN, AK, BK, VEC, E, CE, AMK, BMK><<<p.mt * p.nt * p.splits, 256, T::LDS_BYTES, st>>>(g);
}

template <bool AK, bool BK, bool VEC, class E, class CE, bool AMK, bool BMK>
static void gemm_launch_m(const GemmPlan& p, const GemmArgs& g, hipStream_t st) {
  if (p.bm == 128 && p.bn == 128) gemm_launch_t<128, 128, AK, BK, VEC, E, CE, AMK, BMK>(p, g, st);
  else if (p.bm == 128) gemm_launch_t<128, 64, AK, BK, VEC, E, CE, AMK, BMK>(p, g, st);
  else gemm_launch_t<64, 64, AK, BK, VEC, E, CE, AMK, BMK>(p, g, st);
}

// The masks are template arguments, so that no load or store of the
// staging carries a branch.  The library's products mask only dY: the A
// operand of the data-gradient product (both operands K-contiguous) or
// the B operand of the weight-gradient product (neither).
template <bool AK, bool BK, bool VEC, class E, class CE>
static void gemm_launch(const GemmPlan& p, const GemmArgs& g, hipStream_t st) {
  if constexpr (AK && BK) {
    if (g.amask) { gemm_launch_m<AK, BK, VEC, E, CE, true, false>(p, g, st); return; }
  }
  if constexpr (!AK && !BK) {
    if (g.bmask) { gemm_launch_m<AK, BK, VEC, E, CE, false, true>(p, g, st); return; }
  }
  gemm_launch_m<AK, BK, VEC, E, CE, false, false>(p, g, st);
}

// C (ldc) = epi(A * B): the GEMM applies the epilogue itself when the
// reduction is not split; otherwise it writes per-split partial sums to the
// workspace and gemm_splitk_epilogue adds them in order and applies it.
// colsum (may be null): column sums of B, added by the GEMM when it is not
// split, else by col_sum from (csrc, cmask, cld).
template <bool AK, bool BK, class E, class CE>
static sb_status gemm_run(GemmArgs g, float* ws, size_t ws_bytes, hipStream_t st,
                          const E* csrc = nullptr, const E* cmask = nullptr, int cld = 0) {
  // Masks exist only where gemm_launch instantiates them.
  if ((g.amask && !(AK && BK)) || (g.bmask && (AK || BK))) return SB_ERR_UNSUPPORTED;
  GemmPlan p = gemm_plan(g.M, g.N, g.K, (int)sizeof(E));
  if (p.ws_bytes > 0 && (!ws || ws_bytes < p.ws_bytes)) return SB_ERR_WORKSPACE;
  // Buffer ranges cover whole operands.
  const int64_t a_elems = AK ? (int64_t)(g.M - 1) * g.lda + g.K : (int64_t)(g.K - 1) * g.lda + g.M;
  const int64_t b_elems = BK ? (int64_t)(g.N - 1) * g.ldb + g.K : (int64_t)(g.K - 1) * g.ldb + g.N;
  const int64_t es = (int64_t)sizeof(E);
  if (a_elems * es >= (1ll << 31) || b_elems * es >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  g.mt = p.mt; g.nt = p.nt; g.splits = p.splits; g.k_per_split = p.kps;
  const bool vec = vec_ok<E>(g.a, g.lda, AK ? g.K : g.M) &&
                   vec_ok<E>(g.b, g.ldb, BK ? g.K : g.N) &&
                   (!g.amask || vec_ok<E>(g.amask, g.lda, AK ? g.K : g.M)) &&
                   (!g.bmask || vec_ok<E>(g.bmask, g.ldb, BK ? g.K : g.N)) && p.kps % 4 == 0;
  CE* out = (CE*)g.c;
  const int ldo = g.ldc;
  const float* bias = g.bias;
  const int relu = g.relu, accumulate = g.accumulate;
  float* colsum = g.colsum;
  const int colsum_acc = g.colsum_acc;
  const bool split = p.splits > 1;
  if (split) {
    g.c = ws; g.ldc = g.N;
    g.bias = nullptr; g.relu = 0; g.accumulate = 0;
    g.colsum = nullptr;
  }
  if (vec) gemm_launch<AK, BK, true, E, CE>(p, g, st);
  else gemm_launch<AK, BK, false, E, CE>(p, g, st);
  if (split) {
    const size_t total = (size_t)g.M * g.N;
    gemm_splitk_epilogue<CE><<<(unsigned)((total + 1023) / 1024), 256, 0, st>>>(
        ws, p.splits, g.M, g.N, out, ldo, bias, relu, accumulate);
    if (colsum)
      col_sum<E><<<cdiv(g.N, 64), 1024, 0, st>>>(csrc, cmask, g.K, g.N, cld, colsum,
                                                  colsum_acc);
  }
  return SB_OK;
}

static size_t gemm_ws(int M, int N, int K, int esize) {
  return gemm_plan(M, N, K, esize).ws_bytes;
}

}  // namespace sb

using namespace sb;

static sb_status fc_check(const sb_fc_desc* d) {
  if (!d) return SB_ERR_INVALID_ARG;
  if (d->m <= 0 || d->k_in <= 0 || d->n_shard <= 0) return SB_ERR_INVALID_ARG;
  if (d->ldx < d->k_in || d->ldy < d->n_shard) return SB_ERR_INVALID_ARG;
  if (d->flags & ~SB_FUSE_RELU) return SB_ERR_INVALID_ARG;
  if (d->dtype != SB_F32 && d->dtype != SB_BF16) return SB_ERR_INVALID_ARG;
  return SB_OK;
}

extern "C" size_t sb_fc_workspace_bytes(const sb_fc_desc* d, int pass) {
  if (fc_check(d) != SB_OK) return (size_t)-1;
  const int es = d->dtype == SB_BF16 ? 2 : 4;
  if (pass == SB_FC_FWD) return gemm_ws(d->m, d->n_shard, d->k_in, es);
  if (pass == SB_FC_BWD)   // dX partial, then dW: the two share the workspace
    return std::max(gemm_ws(d->m, d->k_in, d->n_shard, es), gemm_ws(d->k_in, d->n_shard, d->m, es));
  return (size_t)-1;
}

// Forward on operands of type E (fp32, or bf16 bits with a bf16 output).
template <class E>
static sb_status fc_fwd_run(const sb_fc_desc* d, const void* x, const void* w, const float* b,
                            void* y, void* ws, size_t ws_bytes, hipStream_t st) {
  GemmArgs g{};
  g.a = x; g.lda = d->ldx; g.amask = nullptr;
  g.b = w; g.ldb = d->n_shard; g.bmask = nullptr;
  g.c = y; g.ldc = d->ldy;
  g.M = d->m; g.N = d->n_shard; g.K = d->k_in;
  g.bias = b; g.relu = (d->flags & SB_FUSE_RELU) ? 1 : 0; g.accumulate = 0;
  return gemm_run<true, false, E, E>(g, (float*)ws, ws_bytes, st);
}

extern "C" sb_status sb_fc_shard_fwd(const sb_fc_desc* d, const void* x, const void* w,
                                     const float* b, void* y, void* ws, size_t ws_bytes,
                                     void* stream) {
  sb_status s = fc_check(d);
  if (s != SB_OK) return s;
  if (!x || !w || !y) return SB_ERR_INVALID_ARG;
  const size_t es = d->dtype == SB_BF16 ? 2 : 4;
  size_t xb = ((size_t)(d->m - 1) * d->ldx + d->k_in) * es;
  size_t yb = ((size_t)(d->m - 1) * d->ldy + d->n_shard) * es;
  size_t wb = (size_t)d->k_in * d->n_shard * es;
  if (sbh::overlaps(y, yb, x, xb) || sbh::overlaps(y, yb, w, wb) ||
      sbh::overlaps(y, yb, b, b ? d->n_shard * sizeof(float) : 0))
    return SB_ERR_INVALID_ARG;
  // The workspace (split partials) must not overlap any operand.
  const size_t need = sb_fc_workspace_bytes(d, SB_FC_FWD);
  if (need > 0 && (sbh::overlaps(ws, need, x, xb) || sbh::overlaps(ws, need, w, wb) ||
                   sbh::overlaps(ws, need, y, yb) ||
                   sbh::overlaps(ws, need, b, b ? d->n_shard * sizeof(float) : 0)))
    return SB_ERR_INVALID_ARG;
  hipStream_t st = sbh::stream_of(stream);
  s = d->dtype == SB_BF16 ? fc_fwd_run<u16>(d, x, w, b, y, ws, ws_bytes, st)
                          : fc_fwd_run<float>(d, x, w, b, y, ws, ws_bytes, st);
  if (s != SB_OK) return s;
  return sbh::launch_status();
}

// Backward on operands of type E: dx_partial has type E, dW and db fp32.
// db is added up inside the dW product (or by col_sum when that product is
// split).
template <class E>
static sb_status fc_bwd_run(const sb_fc_desc* d, const void* x, const void* w, const void* dy,
                            const void* mask, void* dxp, float* dw, float* db, int accumulate,
                            void* ws, size_t ws_bytes, hipStream_t st) {
  sb_status s;
  if (dxp) {
    GemmArgs g{};
    g.a = dy; g.lda = d->ldy; g.amask = mask;
    g.b = w; g.ldb = d->n_shard; g.bmask = nullptr;
    g.c = dxp; g.ldc = d->ldx;
    g.M = d->m; g.N = d->k_in; g.K = d->n_shard;
    s = gemm_run<true, true, E, E>(g, (float*)ws, ws_bytes, st);
    if (s != SB_OK) return s;
  }
  GemmArgs g{};
  g.a = x; g.lda = d->ldx; g.amask = nullptr;
  g.b = dy; g.ldb = d->ldy; g.bmask = mask;
  g.c = dw; g.ldc = d->n_shard;
  g.M = d->k_in; g.N = d->n_shard; g.K = d->m;
  g.accumulate = accumulate;
  g.colsum = db; g.colsum_acc = accumulate;
  return gemm_run<false, false, E, float>(g, (float*)ws, ws_bytes, st, (const E*)dy,
                                          (const E*)mask, d->ldy);
}

extern "C" sb_status sb_fc_shard_bwd(const sb_fc_desc* d, const void* x, const void* w,
                                     const void* dy, const void* mask, void* dxp, float* dw,
                                     float* db, int accumulate, void* ws, size_t ws_bytes,
                                     void* stream) {
  sb_status s = fc_check(d);
  if (s != SB_OK) return s;
  if (d->flags != 0) return SB_ERR_INVALID_ARG;
  if (!x || !w || !dy || !dw) return SB_ERR_INVALID_ARG;
  if (accumulate != 0 && accumulate != 1) return SB_ERR_INVALID_ARG;
  const size_t es = d->dtype == SB_BF16 ? 2 : 4;
  size_t xb = ((size_t)(d->m - 1) * d->ldx + d->k_in) * es;
  size_t yb = ((size_t)(d->m - 1) * d->ldy + d->n_shard) * es;
  size_t wb = (size_t)d->k_in * d->n_shard * es;
  size_t dwb = (size_t)d->k_in * d->n_shard * sizeof(float);
  size_t dbb = (size_t)d->n_shard * sizeof(float);
  const void* ins[4] = {x, w, dy, mask};
  size_t insb[4] = {xb, wb, yb, mask ? yb : 0};
  void* outs[3] = {dxp, dw, db};
  size_t outsb[3] = {dxp ? xb : 0, dwb, db ? dbb : 0};
  for (int o = 0; o < 3; ++o) {
    for (int i = 0; i < 4; ++i)
      if (sbh::overlaps(outs[o], outsb[o], ins[i], insb[i])) return SB_ERR_INVALID_ARG;
    for (int o2 = o + 1; o2 < 3; ++o2)
      if (sbh::overlaps(outs[o], outsb[o], outs[o2], outsb[o2])) return SB_ERR_INVALID_ARG;
  }
  size_t need = sb_fc_workspace_bytes(d, SB_FC_BWD);
  if (need > 0 && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  // The workspace (split partials) must not overlap any operand.
  if (need > 0) {
    for (int i = 0; i < 4; ++i)
      if (sbh::overlaps(ws, need, ins[i], insb[i])) return SB_ERR_INVALID_ARG;
    for (int o = 0; o < 3; ++o)
      if (sbh::overlaps(ws, need, outs[o], outsb[o])) return SB_ERR_INVALID_ARG;
  }
  hipStream_t st = sbh::stream_of(stream);
  s = d->dtype == SB_BF16
          ? fc_bwd_run<u16>(d, x, w, dy, mask, dxp, dw, db, accumulate, ws, ws_bytes, st)
          : fc_bwd_run<float>(d, x, w, dy, mask, dxp, dw, db, accumulate, ws, ws_bytes, st);
  if (s != SB_OK) return s;
  return sbh::launch_status();
}
