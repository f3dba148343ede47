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
// One fp32 MFMA GEMM kernel serves the three products.  Operands are staged
// in LDS as [k][m] and [k][n] (the MFMA-facing index contiguous) whatever
// their layout in memory: a template flag says whether the global operand is
// contiguous along the reduction index (then the copy into LDS transposes).
// Block tile 128 x 128 x 16, four waves of 64 x 64 (4 x 4 MFMA 16x16 blocks),
// double-buffered global -> register -> LDS pipeline.  When the output tile
// count cannot fill the chip, the reduction is split over gridDim.z and
// gemm_splitk_epilogue sums the splits in a fixed order.
#include "sb_internal.hpp"

#include <algorithm>

namespace sb {

constexpr int GBM = 128, GBN = 128, GBK = 16;
constexpr int GSTR = 128 + 16;         // LDS row stride (floats), = 16 mod 64

struct GemmArgs {
  const float* a; int lda;             // A element (m,k): K_CONTIG ? a[m*lda+k] : a[k*lda+m]
  const float* amask;                  // optional mask, same layout/stride as a
  const float* b; int ldb;             // B element (k,n): K_CONTIG ? b[n*ldb+k] : b[k*ldb+n]
  const float* bmask;
  float* c; int ldc;                   // C[m*ldc + n]
  int M, N, K;
  int k_per_split;
};

template <bool A_KCONTIG, bool B_KCONTIG>
__global__ __launch_bounds__(256, 1) void gemm_f32(GemmArgs g, int partial,
                                                   const float* __restrict__ bias, int relu,
                                                   int accumulate) {
  __shared__ float As[2][GBK * GSTR];
  __shared__ float Bs[2][GBK * GSTR];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int kq = lane >> 4, lr = lane & 15;
  const int m0 = blockIdx.x * GBM, n0 = blockIdx.y * GBN;
  const int kb = blockIdx.z * g.k_per_split;
  const int ke = min(g.K, kb + g.k_per_split);

  f4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  // 2048 elements per operand tile, 8 per thread.
  float ra[8], rb[8];
  auto load_op = [&](const float* p, const float* msk, int ld, bool kcontig, int rows, int r0,
                     int k0, float* r) {
    // Tile element (kk, rr): kk in [0,16), rr in [0,128).
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int e = tid + i * 256;
      int kk, rr;
      if (kcontig) { rr = e / GBK; kk = e - rr * GBK; }   // consecutive threads walk k
      else { kk = e / GBM; rr = e - kk * GBM; }            // consecutive threads walk rows
      int row = r0 + rr, k = k0 + kk;
      bool ok = row < rows && k < ke;
      size_t off = kcontig ? (size_t)row * ld + k : (size_t)k * ld + row;
      float v = ok ? p[off] : 0.f;
      if (msk && ok && !(msk[off] > 0.f)) v = 0.f;
      r[i] = v;
    }
  };
  auto store_op = [&](float* S, bool kcontig, const float* r) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int e = tid + i * 256;
      int kk, rr;
      if (kcontig) { rr = e / GBK; kk = e - rr * GBK; }
      else { kk = e / GBM; rr = e - kk * GBM; }
      S[kk * GSTR + rr] = r[i];
    }
  };

  int nk = cdiv(ke - kb, GBK);
  if (nk > 0) {
    load_op(g.a, g.amask, g.lda, A_KCONTIG, g.M, m0, kb, ra);
    load_op(g.b, g.bmask, g.ldb, B_KCONTIG, g.N, n0, kb, rb);
    store_op(As[0], A_KCONTIG, ra);
    store_op(Bs[0], B_KCONTIG, rb);
  }
  __syncthreads();
  for (int t = 0; t < nk; ++t) {
    const int buf = t & 1;
    const bool more = t + 1 < nk;
    if (more) {
      load_op(g.a, g.amask, g.lda, A_KCONTIG, g.M, m0, kb + (t + 1) * GBK, ra);
      load_op(g.b, g.bmask, g.ldb, B_KCONTIG, g.N, n0, kb + (t + 1) * GBK, rb);
    }
    const float* A = As[buf];
    const float* B = Bs[buf];
#pragma unroll
    for (int ks = 0; ks < GBK / 4; ++ks) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = A[(ks * 4 + kq) * GSTR + wm * 64 + i * 16 + lr];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = B[(ks * 4 + kq) * GSTR + wn * 64 + j * 16 + lr];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x4(av[i], bv[j], acc[i][j]);
    }
    if (more) {
      store_op(As[buf ^ 1], A_KCONTIG, ra);
      store_op(Bs[buf ^ 1], B_KCONTIG, rb);
    }
    __syncthreads();
  }

  // acc[i][j] lane holds C[m0 + wm*64 + i*16 + 4*kq + e][n0 + wn*64 + j*16 + lr].
  float* dst = g.c + (partial ? (size_t)blockIdx.z * g.M * g.ldc : 0);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int m = m0 + wm * 64 + i * 16 + 4 * kq + e;
      if (m >= g.M) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int n = n0 + wn * 64 + j * 16 + lr;
        if (n >= g.N) continue;
        float v = acc[i][j][e];
        size_t o = (size_t)m * g.ldc + n;
        if (!partial) {
          if (bias) v += bias[n];
          if (relu && !(v > 0.f)) v = 0.f;
          if (accumulate) v += dst[o];
        }
        dst[o] = v;
      }
    }
}

// out[m, n] = epi(sum_s part[s][m][n]): + bias[n], ReLU, + out (accumulate).
__global__ __launch_bounds__(256) void gemm_splitk_epilogue(
    const float* __restrict__ part, int splits, int M, int N, int ldp, float* __restrict__ out,
    int ldo, const float* __restrict__ bias, int relu, int accumulate) {
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)M * N) return;
  int m = (int)(i / N), n = (int)(i - (size_t)m * N);
  float v = 0.f;
  for (int s = 0; s < splits; ++s) v += part[((size_t)s * M + m) * ldp + n];
  if (bias) v += bias[n];
  if (relu && !(v > 0.f)) v = 0.f;
  size_t o = (size_t)m * ldo + n;
  if (accumulate) v += out[o];
  out[o] = v;
}

// db[j] = (db[j] +) sum_i G[i][j], rows summed in order.
__global__ __launch_bounds__(256) void col_sum(const float* __restrict__ dy, const float* __restrict__ mask,
                                               int M, int N, int ld, float* __restrict__ db,
                                               int accumulate) {
  int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= N) return;
  float v = 0.f;
  for (int i = 0; i < M; ++i) {
    size_t o = (size_t)i * ld + j;
    float g = dy[o];
    if (mask && !(mask[o] > 0.f)) g = 0.f;
    v += g;
  }
  db[j] = accumulate ? db[j] + v : v;
}

struct GemmPlan { int mt, nt, splits, kps; size_t ws_bytes; };

static GemmPlan gemm_plan(int M, int N, int K) {
  GemmPlan p{};
  p.mt = cdiv(M, GBM);
  p.nt = cdiv(N, GBN);
  long tiles = (long)p.mt * p.nt;
  const long target = 256;
  int splits = 1;
  if (tiles < target) splits = (int)std::min<long>(cdiv(K, GBK), cdiv((int)target, (int)tiles));
  int ktiles = cdiv(K, GBK);
  int tps = cdiv(ktiles, splits);
  p.kps = tps * GBK;
  p.splits = cdiv(K, p.kps);
  p.ws_bytes = p.splits > 1 ? (size_t)p.splits * M * N * sizeof(float) : 0;
  return p;
}

// C (ldc) = epi(A * B): the GEMM applies the epilogue itself when the
// reduction is not split; otherwise it writes per-split partial sums to the
// workspace and gemm_splitk_epilogue adds them in order and applies it.
template <bool AK, bool BK>
static sb_status gemm_run(GemmArgs g, const float* bias, int relu, int accumulate, float* ws,
                          size_t ws_bytes, hipStream_t st) {
  GemmPlan p = gemm_plan(g.M, g.N, g.K);
  if (p.ws_bytes > 0 && (!ws || ws_bytes < p.ws_bytes)) return SB_ERR_WORKSPACE;
  g.k_per_split = p.kps;
  dim3 grid(p.mt, p.nt, p.splits);
  if (p.splits == 1) {
    gemm_f32<AK, BK><<<grid, 256, 0, st>>>(g, 0, bias, relu, accumulate);
    return SB_OK;
  }
  float* out = g.c;
  int ldo = g.ldc;
  g.c = ws;
  g.ldc = g.N;
  gemm_f32<AK, BK><<<grid, 256, 0, st>>>(g, 1, nullptr, 0, 0);
  size_t total = (size_t)g.M * g.N;
  gemm_splitk_epilogue<<<(unsigned)((total + 255) / 256), 256, 0, st>>>(
      ws, p.splits, g.M, g.N, g.N, out, ldo, bias, relu, accumulate);
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
  if (d->dtype == SB_BF16) return SB_ERR_UNSUPPORTED;
  if (d->dtype != SB_F32) return SB_ERR_INVALID_ARG;
  return SB_OK;
}

extern "C" size_t sb_fc_workspace_bytes(const sb_fc_desc* d, int pass) {
  if (fc_check(d) != SB_OK) return (size_t)-1;
  if (pass == SB_FC_FWD) return gemm_ws(d->m, d->n_shard, d->k_in);
  if (pass == SB_FC_BWD)   // dX partial, then dW: the two share the workspace
    return std::max(gemm_ws(d->m, d->k_in, d->n_shard), gemm_ws(d->k_in, d->n_shard, d->m));
  return (size_t)-1;
}

extern "C" sb_status sb_fc_shard_fwd(const sb_fc_desc* d, const void* x, const void* w,
                                     const float* b, void* y, void* ws, size_t ws_bytes,
                                     void* stream) {
  sb_status s = fc_check(d);
  if (s != SB_OK) return s;
  if (!x || !w || !y) return SB_ERR_INVALID_ARG;
  const size_t es = 4;
  size_t xb = ((size_t)(d->m - 1) * d->ldx + d->k_in) * es;
  size_t yb = ((size_t)(d->m - 1) * d->ldy + d->n_shard) * es;
  size_t wb = (size_t)d->k_in * d->n_shard * es;
  if (sbh::overlaps(y, yb, x, xb) || sbh::overlaps(y, yb, w, wb) ||
      sbh::overlaps(y, yb, b, b ? d->n_shard * es : 0))
    return SB_ERR_INVALID_ARG;
  GemmArgs g{};
  g.a = (const float*)x; g.lda = d->ldx; g.amask = nullptr;
  g.b = (const float*)w; g.ldb = d->n_shard; g.bmask = nullptr;
  g.c = (float*)y; g.ldc = d->ldy;
  g.M = d->m; g.N = d->n_shard; g.K = d->k_in;
  hipStream_t st = sbh::stream_of(stream);
  s = gemm_run<true, false>(g, b, (d->flags & SB_FUSE_RELU) ? 1 : 0, 0, (float*)ws, ws_bytes, st);
  if (s != SB_OK) return s;
  return sbh::launch_status();
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
  const size_t es = 4;
  size_t xb = ((size_t)(d->m - 1) * d->ldx + d->k_in) * es;
  size_t yb = ((size_t)(d->m - 1) * d->ldy + d->n_shard) * es;
  size_t wb = (size_t)d->k_in * d->n_shard * es;
  size_t dbb = (size_t)d->n_shard * es;
  const void* ins[4] = {x, w, dy, mask};
  size_t insb[4] = {xb, wb, yb, mask ? yb : 0};
  void* outs[3] = {dxp, dw, db};
  size_t outsb[3] = {dxp ? xb : 0, wb, db ? dbb : 0};
  for (int o = 0; o < 3; ++o) {
    for (int i = 0; i < 4; ++i)
      if (sbh::overlaps(outs[o], outsb[o], ins[i], insb[i])) return SB_ERR_INVALID_ARG;
    for (int o2 = o + 1; o2 < 3; ++o2)
      if (sbh::overlaps(outs[o], outsb[o], outs[o2], outsb[o2])) return SB_ERR_INVALID_ARG;
  }
  size_t need = sb_fc_workspace_bytes(d, SB_FC_BWD);
  if (need > 0 && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  hipStream_t st = sbh::stream_of(stream);
  if (dxp) {
    GemmArgs g{};
    g.a = (const float*)dy; g.lda = d->ldy; g.amask = (const float*)mask;
    g.b = (const float*)w; g.ldb = d->n_shard; g.bmask = nullptr;
    g.c = (float*)dxp; g.ldc = d->ldx;
    g.M = d->m; g.N = d->k_in; g.K = d->n_shard;
    s = gemm_run<true, true>(g, nullptr, 0, 0, (float*)ws, ws_bytes, st);
    if (s != SB_OK) return s;
  }
  {
    GemmArgs g{};
    g.a = (const float*)x; g.lda = d->ldx; g.amask = nullptr;
    g.b = (const float*)dy; g.ldb = d->ldy; g.bmask = (const float*)mask;
    g.c = dw; g.ldc = d->n_shard;
    g.M = d->k_in; g.N = d->n_shard; g.K = d->m;
    s = gemm_run<false, false>(g, nullptr, 0, accumulate, (float*)ws, ws_bytes, st);
    if (s != SB_OK) return s;
  }
  if (db)
    col_sum<<<cdiv(d->n_shard, 256), 256, 0, st>>>((const float*)dy, (const float*)mask, d->m,
                                                   d->n_shard, d->ldy, db, accumulate);
  return sbh::launch_status();
}
