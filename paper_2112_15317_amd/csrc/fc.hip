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
// One fp32 MFMA GEMM kernel serves the three products.  Block tile
// 128 x 128 x 32, four waves of 64 x 64 (4 x 4 MFMA 16x16 blocks).  Each
// operand keeps the layout it has in memory when it is staged in LDS:
//   * contiguous along the reduction index ("K-contiguous"): [row][k], row
//     stride 36 floats; a lane reads 4 consecutive k of its row (16 B), which
//     feed four MFMA k-steps;
//   * contiguous along its row index: [k][row], k stride 132 floats; a lane
//     reads one float per k-step.
// Inside each 16-wide slice of the reduction, MFMA k-step j takes element
// k = 4*kq + j from lane group kq, for both operands, so the two layouts pair
// up (any fixed order of the reduction gives the same sum up to rounding).
// Both layouts are written and read without bank conflicts.  Global loads
// are raw buffer loads whose out-of-range offsets read 0 (nothing waits on
// them until the LDS store); the ReLU mask of dY is applied at that store.
// When the output tiles cannot fill the chip the reduction is split over
// gridDim.z, and gemm_splitk_epilogue sums the splits in a fixed order.
#include "sb_internal.hpp"

#include <algorithm>

namespace sb {

constexpr int GBM = 128, GBN = 128, GBK = 32;
constexpr int RK = GBK + 4;            // [row][k] row stride (floats)
constexpr int RR = GBM + 4;            // [k][row] k stride (floats); 4 * RR = 16 mod 64
constexpr int OPSZ = GBM * RK > GBK * RR ? GBM * RK : GBK * RR;   // floats per operand buffer
constexpr size_t GEMM_LDS_BYTES = 2 * 2 * OPSZ * sizeof(float);    // 2 operands x 2 buffers

// Operands and masks hold elements of the GEMM's operand type E (float or
// bf16 bits), C elements of its output type (or fp32 split partials).
struct GemmArgs {
  const void* a; int lda;              // A element (m,k): A_KC ? a[m*lda+k] : a[k*lda+m]
  const void* amask;                   // optional mask, same layout/stride as a
  const void* b; int ldb;              // B element (k,n): B_KC ? b[n*ldb+k] : b[k*ldb+n]
  const void* bmask;
  void* c; int ldc;                    // C[m*ldc + n]
  int M, N, K;
  int k_per_split;
};

// One operand's staging: 1024 groups of 4 elements per 128 x 32 tile, 4 per
// thread.  K-contiguous: group g = (k quad q = g / 128, row r = g % 128), the
// 4 elements are 4 consecutive k of row r.  Row-contiguous: group g = (k =
// g / 32, row quad = g % 32), the 4 elements are 4 consecutive rows.  VEC
// loads each group with one vector load (aligned, whole groups in range);
// otherwise element by element.  Elements of type E, widened to fp32.
template <bool KC, bool VEC, class E>
struct OpStage {
  f4 v[4];
  __device__ __forceinline__ void load(rsrc_t r, rsrc_t rm, bool masked, int ld, int rows,
                                       int r0, int k0, int ke, int tid) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = tid + i * 256;
      const int row = KC ? r0 + (g & 127) : r0 + (g & 31) * 4;
      const int k = KC ? k0 + (g >> 7) * 4 : k0 + (g >> 5);
      f4 x, m = f4{1.f, 1.f, 1.f, 1.f};
      if (VEC) {
        const bool ok = row < rows && k < ke;       // whole group in range
        const uint32_t off =
            ok ? (uint32_t)(KC ? row * ld + k : k * ld + row) * (uint32_t)sizeof(E) : kOOB;
        x = BufLoad<E>::four(r, off);
        if (masked) m = BufLoad<E>::four(rm, off);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rr = KC ? row : row + e, kk = KC ? k + e : k;
          const bool ok = rr < rows && kk < ke;
          const uint32_t off =
              ok ? (uint32_t)(KC ? rr * ld + kk : kk * ld + rr) * (uint32_t)sizeof(E) : kOOB;
          x[e] = BufLoad<E>::one(r, off);
          if (masked) m[e] = BufLoad<E>::one(rm, off);
        }
      }
      if (masked) {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = m[e] > 0.f ? x[e] : 0.f;
      }
      v[i] = x;
    }
  }
  __device__ __forceinline__ void store(float* S, int tid) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = tid + i * 256;
      float* p = KC ? S + (g & 127) * RK + (g >> 7) * 4 : S + (g >> 5) * RR + (g & 31) * 4;
      *reinterpret_cast<f4*>(p) = v[i];
    }
  }
};

// Operand values of one 16-wide reduction slice for the four 16-row blocks of
// a wave: f[blk][j] = element (row lr of block blk, k = 16*s + 4*kq + j).
template <bool KC>
__device__ __forceinline__ void frag16(const float* S, int row0, int s, int kq, int lr,
                                       f4 (&f)[4]) {
#pragma unroll
  for (int blk = 0; blk < 4; ++blk) {
    const int row = row0 + blk * 16 + lr;
    if (KC) {
      f[blk] = *reinterpret_cast<const f4*>(S + row * RK + s * 16 + kq * 4);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) f[blk][j] = S[(s * 16 + kq * 4 + j) * RR + row];
    }
  }
}

template <bool A_KC, bool B_KC, bool VEC, class E, class CE>
__global__ __launch_bounds__(256, 2) void gemm_f32(GemmArgs g, int partial,
                                                   const float* __restrict__ bias, int relu,
                                                   int accumulate) {
  extern __shared__ float lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int kq = lane >> 4, lr = lane & 15;
  const int m0 = blockIdx.x * GBM, n0 = blockIdx.y * GBN;
  const int kb = blockIdx.z * g.k_per_split;
  const int ke = min(g.K, kb + g.k_per_split);
  // Whole operand tensors (the host keeps them below 2^31 bytes).
  const size_t a_elems = A_KC ? (size_t)(g.M - 1) * g.lda + g.K : (size_t)(g.K - 1) * g.lda + g.M;
  const size_t b_elems = B_KC ? (size_t)(g.N - 1) * g.ldb + g.K : (size_t)(g.K - 1) * g.ldb + g.N;
  const rsrc_t ra = make_rsrc(g.a, (uint32_t)(a_elems * sizeof(E)));
  const rsrc_t rb = make_rsrc(g.b, (uint32_t)(b_elems * sizeof(E)));
  const rsrc_t ram = make_rsrc(g.amask ? g.amask : g.a, (uint32_t)(a_elems * sizeof(E)));
  const rsrc_t rbm = make_rsrc(g.bmask ? g.bmask : g.b, (uint32_t)(b_elems * sizeof(E)));
  const bool amasked = g.amask != nullptr, bmasked = g.bmask != nullptr;

  f4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  OpStage<A_KC, VEC, E> sa;
  OpStage<B_KC, VEC, E> sb_;
  auto Abuf = [&](int b) { return lds + b * 2 * OPSZ; };
  auto Bbuf = [&](int b) { return lds + b * 2 * OPSZ + OPSZ; };

  const int nk = cdiv(ke - kb, GBK);
  if (nk > 0) {
    sa.load(ra, ram, amasked, g.lda, g.M, m0, kb, ke, tid);
    sb_.load(rb, rbm, bmasked, g.ldb, g.N, n0, kb, ke, tid);
    sa.store(Abuf(0), tid);
    sb_.store(Bbuf(0), tid);
    if (nk > 1) {
      sa.load(ra, ram, amasked, g.lda, g.M, m0, kb + GBK, ke, tid);
      sb_.load(rb, rbm, bmasked, g.ldb, g.N, n0, kb + GBK, ke, tid);
    }
  }
  __syncthreads();
  for (int t = 0; t < nk; ++t) {
    const int buf = t & 1;
    if (t + 1 < nk) {
      sa.store(Abuf(buf ^ 1), tid);
      sb_.store(Bbuf(buf ^ 1), tid);
    }
    if (t + 2 < nk) {
      sa.load(ra, ram, amasked, g.lda, g.M, m0, kb + (t + 2) * GBK, ke, tid);
      sb_.load(rb, rbm, bmasked, g.ldb, g.N, n0, kb + (t + 2) * GBK, ke, tid);
    }
    const float* A = Abuf(buf);
    const float* B = Bbuf(buf);
#pragma unroll
    for (int s = 0; s < GBK / 16; ++s) {
      f4 fa[4], fb[4];
      frag16<A_KC>(A, wm * 64, s, kq, lr, fa);
      frag16<B_KC>(B, wn * 64, s, kq, lr, fb);
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int n = 0; n < 4; ++n) acc[i][n] = mfma16x16x4(fa[i][j], fb[n][j], acc[i][n]);
    }
    __syncthreads();
  }

  // acc[i][n] lane holds C[m0 + wm*64 + i*16 + 4*kq + e][n0 + wn*64 + n*16 + lr].
  // Split partials are fp32 (one slab per split); otherwise C has type CE.
  float* part = partial ? (float*)g.c + (size_t)blockIdx.z * g.M * g.ldc : nullptr;
  CE* dst = (CE*)g.c;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int m = m0 + wm * 64 + i * 16 + 4 * kq + e;
      if (m >= g.M) continue;
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        int col = n0 + wn * 64 + n * 16 + lr;
        if (col >= g.N) continue;
        float v = acc[i][n][e];
        size_t o = (size_t)m * g.ldc + col;
        if (partial) {
          part[o] = v;
          continue;
        }
        if (bias) v += bias[col];
        if (relu && !(v > 0.f)) v = 0.f;
        if (accumulate) v += Elem<CE>::load(dst, o);
        Elem<CE>::store(dst, o, v);
      }
    }
}

// out[m, n] = epi(sum_s part[s][m][n]): + bias[n], ReLU, + out (accumulate),
// rounded to the output type CE.
template <class CE>
__global__ __launch_bounds__(256) void gemm_splitk_epilogue(
    const float* __restrict__ part, int splits, int M, int N, int ldp, CE* __restrict__ out,
    int ldo, const float* __restrict__ bias, int relu, int accumulate) {
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)M * N) return;
  int m = (int)(i / N), n = (int)(i - (size_t)m * N);
  float v = 0.f;
  for (int s = 0; s < splits; ++s) v += part[((size_t)s * M + m) * ldp + n];
  if (bias) v += bias[n];
  if (relu && !(v > 0.f)) v = 0.f;
  size_t o = (size_t)m * ldo + n;
  if (accumulate) v += Elem<CE>::load(out, o);
  Elem<CE>::store(out, o, v);
}

// db[j] = (db[j] +) sum_i G[i][j].  A block owns 64 columns; its 16 waves sum
// every 16th row (four independent partial sums each, combined in a fixed
// order), then the wave sums are added in order through LDS.
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

struct GemmPlan { int mt, nt, splits, kps; size_t ws_bytes; };

static GemmPlan gemm_plan(int M, int N, int K) {
  GemmPlan p{};
  p.mt = cdiv(M, GBM);
  p.nt = cdiv(N, GBN);
  long tiles = (long)p.mt * p.nt;
  // About one block per CU, at least two k-tiles per split.
  const long target = 256;
  int ktiles = cdiv(K, GBK);
  int splits = 1;
  if (tiles < target)
    splits = (int)std::min<long>(std::max(1, ktiles / 2), cdiv((int)target, (int)tiles));
  int tps = cdiv(ktiles, splits);
  p.kps = tps * GBK;
  p.splits = cdiv(K, p.kps);
  p.ws_bytes = p.splits > 1 ? (size_t)p.splits * M * N * sizeof(float) : 0;
  return p;
}

// 4-element groups load as one vector (16 bytes fp32, 8 bytes bf16).
template <class E>
static bool vec_ok(const void* p, int ld, int contiguous_extent) {
  return ((uintptr_t)p & (4 * sizeof(E) - 1)) == 0 && ld % 4 == 0 && contiguous_extent % 4 == 0;
}

template <bool AK, bool BK, bool VEC, class E, class CE>
static void gemm_launch(const GemmPlan& p, const GemmArgs& g, int partial, const float* bias,
                        int relu, int accumulate, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)gemm_f32<AK, BK, VEC, E, CE>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)GEMM_LDS_BYTES);
    attr_set = true;
  }
  dim3 grid(p.mt, p.nt, p.splits);
  gemm_f32<AK, BK, VEC, E, CE><<<grid, 256, GEMM_LDS_BYTES, st>>>(g, partial, bias, relu,
                                                                   accumulate);
}

// C (ldc) = epi(A * B): the GEMM applies the epilogue itself when the
// reduction is not split; otherwise it writes per-split partial sums to the
// workspace and gemm_splitk_epilogue adds them in order and applies it.
template <bool AK, bool BK, class E, class CE>
static sb_status gemm_run(GemmArgs g, const float* bias, int relu, int accumulate, float* ws,
                          size_t ws_bytes, hipStream_t st) {
  GemmPlan p = gemm_plan(g.M, g.N, g.K);
  if (p.ws_bytes > 0 && (!ws || ws_bytes < p.ws_bytes)) return SB_ERR_WORKSPACE;
  // Buffer ranges cover whole operands.
  const int64_t a_elems = AK ? (int64_t)(g.M - 1) * g.lda + g.K : (int64_t)(g.K - 1) * g.lda + g.M;
  const int64_t b_elems = BK ? (int64_t)(g.N - 1) * g.ldb + g.K : (int64_t)(g.K - 1) * g.ldb + g.N;
  const int64_t es = (int64_t)sizeof(E);
  if (a_elems * es >= (1ll << 31) || b_elems * es >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  g.k_per_split = p.kps;
  const bool vec = vec_ok<E>(g.a, g.lda, AK ? g.K : g.M) &&
                   vec_ok<E>(g.b, g.ldb, BK ? g.K : g.N) &&
                   (!g.amask || vec_ok<E>(g.amask, g.lda, AK ? g.K : g.M)) &&
                   (!g.bmask || vec_ok<E>(g.bmask, g.ldb, BK ? g.K : g.N)) && p.kps % 4 == 0;
  CE* out = (CE*)g.c;
  int ldo = g.ldc;
  const bool split = p.splits > 1;
  if (split) { g.c = ws; g.ldc = g.N; }
  if (vec) gemm_launch<AK, BK, true, E, CE>(p, g, split, split ? nullptr : bias,
                                            split ? 0 : relu, split ? 0 : accumulate, st);
  else gemm_launch<AK, BK, false, E, CE>(p, g, split, split ? nullptr : bias, split ? 0 : relu,
                                         split ? 0 : accumulate, st);
  if (split) {
    size_t total = (size_t)g.M * g.N;
    gemm_splitk_epilogue<CE><<<(unsigned)((total + 255) / 256), 256, 0, st>>>(
        ws, p.splits, g.M, g.N, g.N, out, ldo, bias, relu, accumulate);
  }
  return SB_OK;
}

static size_t gemm_ws(int M, int N, int K) { return gemm_plan(M, N, K).ws_bytes; }

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
  if (pass == SB_FC_FWD) return gemm_ws(d->m, d->n_shard, d->k_in);
  if (pass == SB_FC_BWD)   // dX partial, then dW: the two share the workspace
    return std::max(gemm_ws(d->m, d->k_in, d->n_shard), gemm_ws(d->k_in, d->n_shard, d->m));
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
  return gemm_run<true, false, E, E>(g, b, (d->flags & SB_FUSE_RELU) ? 1 : 0, 0, (float*)ws,
                                     ws_bytes, st);
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
    s = gemm_run<true, true, E, E>(g, nullptr, 0, 0, (float*)ws, ws_bytes, st);
    if (s != SB_OK) return s;
  }
  {
    GemmArgs g{};
    g.a = x; g.lda = d->ldx; g.amask = nullptr;
    g.b = dy; g.ldb = d->ldy; g.bmask = mask;
    g.c = dw; g.ldc = d->n_shard;
    g.M = d->k_in; g.N = d->n_shard; g.K = d->m;
    s = gemm_run<false, false, E, float>(g, nullptr, 0, accumulate, (float*)ws, ws_bytes, st);
    if (s != SB_OK) return s;
  }
  if (db)
    col_sum<E><<<cdiv(d->n_shard, 64), 1024, 0, st>>>((const E*)dy, (const E*)mask, d->m,
                                                      d->n_shard, d->ldy, db, accumulate);
  return SB_OK;
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
