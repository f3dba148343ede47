// api.hip -- the convolution entry points of libsb: argument validation,
// workspace sizing and dispatch to the kernels.  Nothing is enqueued unless
// every check passes.
#include "conv_common.hpp"

#include <mutex>

namespace sbh {
int conv_igemm_pack_task(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout,
                         const void* wt, void* packed, sb::PackTask* t);
void conv_pack_many(int dtype, const sb::PackBatch& b, hipStream_t st);
size_t conv_igemm_ws(int dtype, int N, int Cin, int H, int W, int Cout, bool prepacked);
size_t conv_igemm_pack_bytes(int dtype, int N, int Cin, int H, int W, int Cout);
void conv_igemm_pack(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout,
                     const void* wt, void* packed, hipStream_t st);
sb_status conv_igemm(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout,
                     const void* in, const void* wt, const float* bias, const void* mask,
                     void* out, void* ws, size_t ws_bytes, int relu, bool prepacked,
                     hipStream_t st, uint8_t* pool_idx = nullptr);
bool conv_igemm_pools(int dtype, int N, int Cin, int H, int W, int Cout);
size_t conv_wgrad_ws(int dtype, int N, int C, int H, int W, int K);
int conv_igemm_describe(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout, char* buf,
                        size_t len, bool pool = false);
int conv_wgrad_describe(int dtype, int N, int C, int H, int W, int K, char* buf, size_t len);
sb_status conv_wgrad(int dtype, int N, int C, int H, int W, int K, const void* x, const void* dy,
                     float* dw, float* db, void* ws, size_t ws_bytes, hipStream_t st);
int conv_wgrad_batch_key(int dtype, int N, int C, int H, int W, int K, const void* x,
                         const void* dy);
sb_status conv_wgrad_group(int n, const int (*shape)[5], const void* const* x,
                           const void* const* dy, float* const* dw, float* const* db,
                           void* const* ws, const size_t* ws_bytes, hipStream_t st);
// Channel-blocked bf16 (SB_NCHW8C).
bool conv_bf16_takes(int N, int Cin, int H, int W, int Cout);
int conv_bf16c8_describe(bool dgrad, int N, int Cin, int H, int W, int Cout, char* buf,
                         size_t len, bool pool = false);
bool conv_bf16c8_pools(int N, int Cin, int H, int W, int Cout);
sb_status conv_bf16c8(bool dgrad, int N, int Cin, int H, int W, int Cout, const void* in,
                      const void* wt, const float* bias, const void* mask, void* out, void* ws,
                      size_t ws_bytes, int relu, bool prepacked, hipStream_t st,
                      uint8_t* pool_idx = nullptr);
bool conv_wgrad_c8_takes(int N, int C, int H, int W, int K);
size_t conv_wgrad_c8_ws(int N, int C, int H, int W, int K);
int conv_wgrad_c8_describe(int N, int C, int H, int W, int K, char* buf, size_t len);
sb_status conv_wgrad_c8(int N, int C, int H, int W, int K, const void* x, const void* dy,
                        float* dw, float* db, void* ws, size_t ws_bytes, hipStream_t st);
}  // namespace sbh

extern "C" const char* sb_status_string(sb_status s) {
  switch (s) {
    case SB_OK: return "SB_OK";
    case SB_ERR_INVALID_ARG: return "SB_ERR_INVALID_ARG";
    case SB_ERR_UNSUPPORTED: return "SB_ERR_UNSUPPORTED";
    case SB_ERR_WORKSPACE: return "SB_ERR_WORKSPACE";
    case SB_ERR_HIP: return "SB_ERR_HIP";
  }
  return "SB_ERR_UNKNOWN";
}

extern "C" int sb_version(void) { return 100; }

static sb_status conv_check(const sb_conv3x3_desc* d, int pass) {
  if (!d) return SB_ERR_INVALID_ARG;
  if (d->n <= 0 || d->c <= 0 || d->h <= 0 || d->w <= 0 || d->k <= 0) return SB_ERR_INVALID_ARG;
  if (d->dtype != SB_F32 && d->dtype != SB_BF16) return SB_ERR_INVALID_ARG;
  if (d->flags & ~(SB_FUSE_RELU | SB_PACKED_FILTERS)) return SB_ERR_INVALID_ARG;
  if (pass != SB_PASS_FWD && (d->flags & SB_FUSE_RELU)) return SB_ERR_INVALID_ARG;
  if (pass == SB_PASS_BWD_WEIGHT && d->flags) return SB_ERR_INVALID_ARG;
  if (d->layout != SB_NCHW && d->layout != SB_NCHW8C) return SB_ERR_INVALID_ARG;
  if (d->layout == SB_NCHW8C) {
    // Channel-blocked tensors: whole 8-channel blocks, on the bf16 MFMA
    // kernels (images at least 8 wide).
    if (d->c % 8 || d->k % 8) return SB_ERR_INVALID_ARG;
    if (d->dtype != SB_BF16) return SB_ERR_UNSUPPORTED;
    const bool ok = pass == SB_PASS_BWD_WEIGHT
                        ? sbh::conv_wgrad_c8_takes(d->n, d->c, d->h, d->w, d->k)
                    : pass == SB_PASS_BWD_DATA
                        ? sbh::conv_bf16_takes(d->n, d->k, d->h, d->w, d->c)
                        : sbh::conv_bf16_takes(d->n, d->c, d->h, d->w, d->k);
    if (!ok) return SB_ERR_UNSUPPORTED;
  }
  if (pass == SB_PASS_FWD_POOL) {
    // Forward with fused ReLU + 2x2 pooling: channel-blocked bf16 or NCHW
    // fp32, even image sizes, an unsplit channel loop.
    if (d->h % 2 || d->w % 2) return SB_ERR_INVALID_ARG;
    const bool ok = d->layout == SB_NCHW8C
                        ? sbh::conv_bf16c8_pools(d->n, d->c, d->h, d->w, d->k)
                        : sbh::conv_igemm_pools(d->dtype, d->n, d->c, d->h, d->w, d->k);
    if (!ok) return SB_ERR_UNSUPPORTED;
  }
  // Kernels index weights and activations with 32-bit ints.
  if ((int64_t)d->k * d->c * 9 >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  if ((int64_t)d->n * d->c * d->h * d->w >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  if ((int64_t)d->n * d->k * d->h * d->w >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  return SB_OK;
}

// Split-partial bytes of a weight-gradient call (the kernel depends on the layout).
static size_t wgrad_ws(const sb_conv3x3_desc* d) {
  return d->layout == SB_NCHW8C ? sbh::conv_wgrad_c8_ws(d->n, d->c, d->h, d->w, d->k)
                                : sbh::conv_wgrad_ws(d->dtype, d->n, d->c, d->h, d->w, d->k);
}

extern "C" size_t sb_conv3x3_workspace_bytes(const sb_conv3x3_desc* d, int pass) {
  if (pass < SB_PASS_FWD || pass > SB_PASS_FWD_POOL) return (size_t)-1;
  if (conv_check(d, pass) != SB_OK) return (size_t)-1;
  const bool pk = (d->flags & SB_PACKED_FILTERS) != 0;
  switch (pass) {
    case SB_PASS_FWD:
    case SB_PASS_FWD_POOL: return sbh::conv_igemm_ws(d->dtype, d->n, d->c, d->h, d->w, d->k, pk);
    case SB_PASS_BWD_DATA: return sbh::conv_igemm_ws(d->dtype, d->n, d->k, d->h, d->w, d->c, pk);
    default: return wgrad_ws(d);
  }
}

// Packed-filter bytes of a forward or data-gradient pass (0: invalid).
static size_t packed_bytes(const sb_conv3x3_desc* d, int pass) {
  if (pass == SB_PASS_FWD || pass == SB_PASS_FWD_POOL) return sbh::conv_igemm_pack_bytes(d->dtype, d->n, d->c, d->h, d->w, d->k);
  return sbh::conv_igemm_pack_bytes(d->dtype, d->n, d->k, d->h, d->w, d->c);
}

extern "C" size_t sb_conv3x3_packed_bytes(const sb_conv3x3_desc* d, int pass) {
  if (pass != SB_PASS_FWD && pass != SB_PASS_BWD_DATA) return 0;
  if (!d) return 0;
  sb_conv3x3_desc q = *d;
  q.flags = 0;
  if (conv_check(&q, pass) != SB_OK) return 0;
  return packed_bytes(&q, pass);
}

extern "C" sb_status sb_conv3x3_pack_filters(const sb_conv3x3_desc* d, int pass, const void* w,
                                             void* packed, size_t packed_bytes_, void* stream) {
  if (pass != SB_PASS_FWD && pass != SB_PASS_BWD_DATA) return SB_ERR_INVALID_ARG;
  if (!d) return SB_ERR_INVALID_ARG;
  sb_conv3x3_desc q = *d;
  q.flags = 0;
  sb_status s = conv_check(&q, pass);
  if (s != SB_OK) return s;
  if (!w || !packed) return SB_ERR_INVALID_ARG;
  const size_t need = packed_bytes(&q, pass);
  const size_t wb = (size_t)q.k * q.c * 9 * sbh::dsize(q.dtype);
  if (packed_bytes_ < need || sbh::overlaps(w, wb, packed, need)) return SB_ERR_INVALID_ARG;
  if (pass == SB_PASS_FWD)
    sbh::conv_igemm_pack(false, q.dtype, q.n, q.c, q.h, q.w, q.k, w, packed,
                         sbh::stream_of(stream));
  else
    sbh::conv_igemm_pack(true, q.dtype, q.n, q.k, q.h, q.w, q.c, w, packed,
                         sbh::stream_of(stream));
  return sbh::launch_status();
}

static size_t act_bytes(const sb_conv3x3_desc* d, int ch) {
  return (size_t)d->n * ch * d->h * d->w * sbh::dsize(d->dtype);
}

extern "C" sb_status sb_conv3x3_pack_filters_many(int count, const sb_conv3x3_desc* descs,
                                                  const int* passes, const void* const* w,
                                                  void* const* packed,
                                                  const size_t* packed_bytes_, void* stream) {
  if (count <= 0 || count > sb::kMaxPackTasks || !descs || !passes || !w || !packed ||
      !packed_bytes_)
    return SB_ERR_INVALID_ARG;
  sb::PackBatch b{};
  b.ntasks = count;
  b.block0[0] = 0;
  for (int i = 0; i < count; ++i) {
    const int pass = passes[i];
    if (pass != SB_PASS_FWD && pass != SB_PASS_BWD_DATA) return SB_ERR_INVALID_ARG;
    sb_conv3x3_desc q = descs[i];
    q.flags = 0;
    sb_status s = conv_check(&q, pass);
    if (s != SB_OK) return s;
    if (q.dtype != descs[0].dtype) return SB_ERR_INVALID_ARG;
    if (!w[i] || !packed[i]) return SB_ERR_INVALID_ARG;
    const size_t need = packed_bytes(&q, pass);
    const size_t wb = (size_t)q.k * q.c * 9 * sbh::dsize(q.dtype);
    if (packed_bytes_[i] < need || sbh::overlaps(w[i], wb, packed[i], need))
      return SB_ERR_INVALID_ARG;
    // Packed outputs must not overlap one another, nor any task's source
    // filters (all tasks run in one launch).
    for (int j = 0; j < i; ++j)
      if (sbh::overlaps(packed[j], packed_bytes_[j], packed[i], need)) return SB_ERR_INVALID_ARG;
    for (int j = 0; j < count; ++j) {
      if (!w[j]) return SB_ERR_INVALID_ARG;
      const size_t wbj = (size_t)descs[j].k * descs[j].c * 9 * sbh::dsize(descs[j].dtype);
      if (sbh::overlaps(w[j], wbj, packed[i], need)) return SB_ERR_INVALID_ARG;
    }
    const int slices =
        pass == SB_PASS_FWD
            ? sbh::conv_igemm_pack_task(false, q.dtype, q.n, q.c, q.h, q.w, q.k, w[i], packed[i],
                                        &b.t[i])
            : sbh::conv_igemm_pack_task(true, q.dtype, q.n, q.k, q.h, q.w, q.c, w[i], packed[i],
                                        &b.t[i]);
    if ((int64_t)b.block0[i] + slices >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
    b.block0[i + 1] = b.block0[i] + slices;
  }
  sbh::conv_pack_many(descs[0].dtype, b, sbh::stream_of(stream));
  return sbh::launch_status();
}

extern "C" sb_status sb_conv3x3_fwd(const sb_conv3x3_desc* d, const void* x, const void* w,
                                    const float* bias, void* y, void* ws, size_t ws_bytes,
                                    void* stream) {
  sb_status s = conv_check(d, SB_PASS_FWD);
  if (s != SB_OK) return s;
  if (!x || !w || !y) return SB_ERR_INVALID_ARG;
  const bool pk = (d->flags & SB_PACKED_FILTERS) != 0;
  size_t yb = act_bytes(d, d->k), xb = act_bytes(d, d->c);
  size_t wb = pk ? packed_bytes(d, SB_PASS_FWD) : (size_t)d->k * d->c * 9 * sbh::dsize(d->dtype);
  if (sbh::overlaps(y, yb, x, xb) || sbh::overlaps(y, yb, w, wb) ||
      sbh::overlaps(y, yb, bias, bias ? d->k * sizeof(float) : 0))
    return SB_ERR_INVALID_ARG;
  size_t need = sbh::conv_igemm_ws(d->dtype, d->n, d->c, d->h, d->w, d->k, pk);
  if (need && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  if (need && (sbh::overlaps(ws, need, x, xb) || sbh::overlaps(ws, need, y, yb) ||
               sbh::overlaps(ws, need, w, wb) ||
               sbh::overlaps(ws, need, bias, bias ? d->k * sizeof(float) : 0)))
    return SB_ERR_INVALID_ARG;
  if (d->layout == SB_NCHW8C)
    return sbh::conv_bf16c8(false, d->n, d->c, d->h, d->w, d->k, x, w, bias, nullptr, y, ws,
                            ws_bytes, (d->flags & SB_FUSE_RELU) ? 1 : 0, pk,
                            sbh::stream_of(stream));
  return sbh::conv_igemm(false, d->dtype, d->n, d->c, d->h, d->w, d->k, x, w, bias, nullptr, y,
                         ws, ws_bytes, (d->flags & SB_FUSE_RELU) ? 1 : 0, pk,
                         sbh::stream_of(stream));
}

extern "C" sb_status sb_conv3x3_fwd_pool(const sb_conv3x3_desc* d, const void* x, const void* w,
                                         const float* bias, void* y, uint8_t* idx, void* ws,
                                         size_t ws_bytes, void* stream) {
  sb_status s = conv_check(d, SB_PASS_FWD_POOL);
  if (s != SB_OK) return s;
  if (!x || !w || !y || !idx) return SB_ERR_INVALID_ARG;
  const bool pk = (d->flags & SB_PACKED_FILTERS) != 0;
  const size_t pooled = (size_t)d->n * d->k * (d->h / 2) * (d->w / 2);
  const size_t yb = pooled * sbh::dsize(d->dtype), ib = pooled, xb = act_bytes(d, d->c);
  const size_t wb = pk ? packed_bytes(d, SB_PASS_FWD) : (size_t)d->k * d->c * 9 * sbh::dsize(d->dtype);
  const size_t bb = bias ? d->k * sizeof(float) : 0;
  if (sbh::overlaps(y, yb, x, xb) || sbh::overlaps(y, yb, w, wb) || sbh::overlaps(y, yb, bias, bb) ||
      sbh::overlaps(idx, ib, x, xb) || sbh::overlaps(idx, ib, w, wb) ||
      sbh::overlaps(idx, ib, bias, bb) || sbh::overlaps(idx, ib, y, yb))
    return SB_ERR_INVALID_ARG;
  size_t need = sbh::conv_igemm_ws(d->dtype, d->n, d->c, d->h, d->w, d->k, pk);
  if (need && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  if (need && (sbh::overlaps(ws, need, x, xb) || sbh::overlaps(ws, need, y, yb) ||
               sbh::overlaps(ws, need, idx, ib) || sbh::overlaps(ws, need, w, wb) ||
               sbh::overlaps(ws, need, bias, bb)))
    return SB_ERR_INVALID_ARG;
  if (d->layout == SB_NCHW8C)
    return sbh::conv_bf16c8(false, d->n, d->c, d->h, d->w, d->k, x, w, bias, nullptr, y, ws,
                            ws_bytes, 0, pk, sbh::stream_of(stream), idx);
  return sbh::conv_igemm(false, d->dtype, d->n, d->c, d->h, d->w, d->k, x, w, bias, nullptr, y,
                         ws, ws_bytes, 0, pk, sbh::stream_of(stream), idx);
}

extern "C" sb_status sb_conv3x3_bwd_data(const sb_conv3x3_desc* d, const void* dy, const void* w,
                                         const void* mask, void* dx, void* ws, size_t ws_bytes,
                                         void* stream) {
  sb_status s = conv_check(d, SB_PASS_BWD_DATA);
  if (s != SB_OK) return s;
  if (!dy || !w || !dx) return SB_ERR_INVALID_ARG;
  const bool pk = (d->flags & SB_PACKED_FILTERS) != 0;
  size_t dxb = act_bytes(d, d->c), dyb = act_bytes(d, d->k);
  size_t wb =
      pk ? packed_bytes(d, SB_PASS_BWD_DATA) : (size_t)d->k * d->c * 9 * sbh::dsize(d->dtype);
  if (sbh::overlaps(dx, dxb, dy, dyb) || sbh::overlaps(dx, dxb, w, wb) ||
      sbh::overlaps(dx, dxb, mask, mask ? dxb : 0))
    return SB_ERR_INVALID_ARG;
  size_t need = sbh::conv_igemm_ws(d->dtype, d->n, d->k, d->h, d->w, d->c, pk);
  if (need && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  if (need && (sbh::overlaps(ws, need, dy, dyb) || sbh::overlaps(ws, need, dx, dxb) ||
               sbh::overlaps(ws, need, w, wb) ||
               sbh::overlaps(ws, need, mask, mask ? dxb : 0)))
    return SB_ERR_INVALID_ARG;
  if (d->layout == SB_NCHW8C)
    return sbh::conv_bf16c8(true, d->n, d->k, d->h, d->w, d->c, dy, w, nullptr, mask, dx, ws,
                            ws_bytes, 0, pk, sbh::stream_of(stream));
  return sbh::conv_igemm(true, d->dtype, d->n, d->k, d->h, d->w, d->c, dy, w, nullptr, mask, dx,
                         ws, ws_bytes, 0, pk, sbh::stream_of(stream));
}

extern "C" sb_status sb_conv3x3_bwd_weight(const sb_conv3x3_desc* d, const void* x, const void* dy,
                                           float* dw, float* db, void* ws, size_t ws_bytes,
                                           void* stream) {
  sb_status s = conv_check(d, SB_PASS_BWD_WEIGHT);
  if (s != SB_OK) return s;
  if (!x || !dy || !dw) return SB_ERR_INVALID_ARG;
  size_t xb = act_bytes(d, d->c), dyb = act_bytes(d, d->k);
  size_t dwb = (size_t)d->k * d->c * 9 * sizeof(float), dbb = db ? d->k * sizeof(float) : 0;
  if (sbh::overlaps(dw, dwb, x, xb) || sbh::overlaps(dw, dwb, dy, dyb) ||
      sbh::overlaps(db, dbb, x, xb) || sbh::overlaps(db, dbb, dy, dyb) ||
      sbh::overlaps(dw, dwb, db, dbb))
    return SB_ERR_INVALID_ARG;
  size_t need = wgrad_ws(d);
  if (need && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  if (need && (sbh::overlaps(ws, need, dw, dwb) || sbh::overlaps(ws, need, db, dbb) ||
               sbh::overlaps(ws, need, x, xb) || sbh::overlaps(ws, need, dy, dyb)))
    return SB_ERR_INVALID_ARG;
  if (d->layout == SB_NCHW8C)
    return sbh::conv_wgrad_c8(d->n, d->c, d->h, d->w, d->k, x, dy, dw, db, ws, ws_bytes,
                              sbh::stream_of(stream));
  return sbh::conv_wgrad(d->dtype, d->n, d->c, d->h, d->w, d->k, x, dy, dw, db, ws, ws_bytes,
                         sbh::stream_of(stream));
}

// ---------------------------------------------------------------------------
// Weight gradients of several layers.  Layer i's split partials live in its
// own region of the workspace (regions in layer order, each rounded up to
// 256 bytes), so the layers need not run one after another: consecutive
// layers whose plans run the same kernel instantiation share one launch.
namespace {
constexpr int kWgGroup = 4;          // layers per shared launch

size_t wgrad_region(const sb_conv3x3_desc* d) { return (wgrad_ws(d) + 255) / 256 * 256; }
}  // namespace

extern "C" size_t sb_conv3x3_bwd_weight_many_workspace_bytes(int count,
                                                             const sb_conv3x3_desc* descs) {
  if (count < 1 || count > SB_MANY_MAX || !descs) return (size_t)-1;
  size_t total = 0;
  for (int i = 0; i < count; ++i) {
    if (conv_check(&descs[i], SB_PASS_BWD_WEIGHT) != SB_OK) return (size_t)-1;
    total += wgrad_region(&descs[i]);
  }
  return total;
}

extern "C" sb_status sb_conv3x3_bwd_weight_many(int count, const sb_conv3x3_desc* d,
                                                const void* const* x, const void* const* dy,
                                                float* const* dw, float* const* db, void* ws,
                                                size_t ws_bytes, void* stream) {
  if (count < 1 || count > SB_MANY_MAX || !d || !x || !dy || !dw) return SB_ERR_INVALID_ARG;
  size_t xb[SB_MANY_MAX], dyb[SB_MANY_MAX], dwb[SB_MANY_MAX], dbb[SB_MANY_MAX];
  size_t off[SB_MANY_MAX + 1];
  off[0] = 0;
  for (int i = 0; i < count; ++i) {
    sb_status s = conv_check(&d[i], SB_PASS_BWD_WEIGHT);
    if (s != SB_OK) return s;
    if (!x[i] || !dy[i] || !dw[i]) return SB_ERR_INVALID_ARG;
    xb[i] = act_bytes(&d[i], d[i].c);
    dyb[i] = act_bytes(&d[i], d[i].k);
    dwb[i] = (size_t)d[i].k * d[i].c * 9 * sizeof(float);
    dbb[i] = db && db[i] ? d[i].k * sizeof(float) : 0;
    off[i + 1] = off[i] + wgrad_region(&d[i]);
  }
  const float* dbp[SB_MANY_MAX];
  for (int i = 0; i < count; ++i) dbp[i] = db ? db[i] : nullptr;
  // No output may overlap any layer's inputs or any other output.
  for (int i = 0; i < count; ++i) {
    if (sbh::overlaps(dw[i], dwb[i], dbp[i], dbb[i])) return SB_ERR_INVALID_ARG;
    for (int j = 0; j < count; ++j) {
      if (sbh::overlaps(dw[i], dwb[i], x[j], xb[j]) || sbh::overlaps(dw[i], dwb[i], dy[j], dyb[j]) ||
          sbh::overlaps(dbp[i], dbb[i], x[j], xb[j]) || sbh::overlaps(dbp[i], dbb[i], dy[j], dyb[j]))
        return SB_ERR_INVALID_ARG;
      if (j != i && (sbh::overlaps(dw[i], dwb[i], dw[j], dwb[j]) ||
                     sbh::overlaps(dw[i], dwb[i], dbp[j], dbb[j]) ||
                     sbh::overlaps(dbp[i], dbb[i], dbp[j], dbb[j])))
        return SB_ERR_INVALID_ARG;
    }
  }
  const size_t need = off[count];
  if (need && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  if (need)
    for (int j = 0; j < count; ++j)
      if (sbh::overlaps(ws, need, x[j], xb[j]) || sbh::overlaps(ws, need, dy[j], dyb[j]) ||
          sbh::overlaps(ws, need, dw[j], dwb[j]) || sbh::overlaps(ws, need, dbp[j], dbb[j]))
        return SB_ERR_INVALID_ARG;
  hipStream_t st = sbh::stream_of(stream);
  char* wsc = (char*)ws;
  auto key_of = [&](int i) {
    return d[i].layout == SB_NCHW8C
               ? -1
               : sbh::conv_wgrad_batch_key(d[i].dtype, d[i].n, d[i].c, d[i].h, d[i].w, d[i].k,
                                           x[i], dy[i]);
  };
  int i = 0;
  while (i < count) {
    const int key = key_of(i);
    sb_status s;
    if (key < 0) {
      void* wsi = need ? wsc + off[i] : nullptr;
      const size_t wsb = off[i + 1] - off[i];
      s = d[i].layout == SB_NCHW8C
              ? sbh::conv_wgrad_c8(d[i].n, d[i].c, d[i].h, d[i].w, d[i].k, x[i], dy[i], dw[i],
                                   dbp[i] ? (float*)dbp[i] : nullptr, wsi, wsb, st)
              : sbh::conv_wgrad(d[i].dtype, d[i].n, d[i].c, d[i].h, d[i].w, d[i].k, x[i], dy[i],
                                dw[i], dbp[i] ? (float*)dbp[i] : nullptr, wsi, wsb, st);
      if (s != SB_OK) return s;
      ++i;
      continue;
    }
    int j = i + 1;
    while (j < count && j - i < kWgGroup && key_of(j) == key) ++j;
    int shape[kWgGroup][5];
    const void* xs[kWgGroup];
    const void* dys[kWgGroup];
    float* dws[kWgGroup];
    float* dbs[kWgGroup];
    void* wss[kWgGroup];
    size_t wsbs[kWgGroup];
    for (int t = i; t < j; ++t) {
      const int u = t - i;
      shape[u][0] = d[t].n; shape[u][1] = d[t].c; shape[u][2] = d[t].h;
      shape[u][3] = d[t].w; shape[u][4] = d[t].k;
      xs[u] = x[t]; dys[u] = dy[t]; dws[u] = dw[t];
      dbs[u] = dbp[t] ? (float*)dbp[t] : nullptr;
      wss[u] = need ? wsc + off[t] : nullptr;
      wsbs[u] = off[t + 1] - off[t];
    }
    s = sbh::conv_wgrad_group(j - i, shape, xs, dys, dws, dbs, wss, wsbs, st);
    if (s != SB_OK) return s;
    i = j;
  }
  return sbh::launch_status();
}

// ---------------------------------------------------------------------------
// Weight gradient without allocation: the split partial sums go to a scratch
// array that the library holds in device memory.  `scratch` is a host-side
// stand-in in host code: its device address is looked up once per device
// (hipGetSymbolAddress, with that device current) and only that address is
// ever handed to a kernel.
namespace {
constexpr size_t kScratchBytes = (size_t)SB_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array.
sb_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SB_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SB_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return SB_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SB_OK;
}
}  // namespace

extern "C" sb_status sb_conv3x3_bwd_weight_noalloc(const sb_conv3x3_desc* d, const void* x,
                                                   const void* dy, float* dw, float* db,
                                                   void* stream) {
  sb_status s = conv_check(d, SB_PASS_BWD_WEIGHT);
  if (s != SB_OK) return s;
  if (!x || !dy || !dw) return SB_ERR_INVALID_ARG;
  size_t xb = act_bytes(d, d->c), dyb = act_bytes(d, d->k);
  size_t dwb = (size_t)d->k * d->c * 9 * sizeof(float), dbb = db ? d->k * sizeof(float) : 0;
  if (sbh::overlaps(dw, dwb, x, xb) || sbh::overlaps(dw, dwb, dy, dyb) ||
      sbh::overlaps(db, dbb, x, xb) || sbh::overlaps(db, dbb, dy, dyb) ||
      sbh::overlaps(dw, dwb, db, dbb))
    return SB_ERR_INVALID_ARG;
  const size_t need = wgrad_ws(d);
  if (need > kScratchBytes) return SB_ERR_WORKSPACE;
  void* ws = nullptr;
  s = scratch_address(&ws);
  if (s != SB_OK) return s;
  if (need && (sbh::overlaps(ws, need, dw, dwb) || sbh::overlaps(ws, need, db, dbb) ||
               sbh::overlaps(ws, need, x, xb) || sbh::overlaps(ws, need, dy, dyb)))
    return SB_ERR_INVALID_ARG;
  if (d->layout == SB_NCHW8C)
    return sbh::conv_wgrad_c8(d->n, d->c, d->h, d->w, d->k, x, dy, dw, db, ws, kScratchBytes,
                              sbh::stream_of(stream));
  return sbh::conv_wgrad(d->dtype, d->n, d->c, d->h, d->w, d->k, x, dy, dw, db, ws,
                         kScratchBytes, sbh::stream_of(stream));
}

extern "C" size_t sb_conv3x3_plan_string(const sb_conv3x3_desc* d, int pass, char* buf,
                                         size_t len) {
  if (pass < SB_PASS_FWD || pass > SB_PASS_FWD_POOL) return 0;
  if (conv_check(d, pass) != SB_OK) return 0;
  int r;
  if (d->layout == SB_NCHW8C) {
    if (pass == SB_PASS_FWD || pass == SB_PASS_FWD_POOL)
      r = sbh::conv_bf16c8_describe(false, d->n, d->c, d->h, d->w, d->k, buf, len,
                                    pass == SB_PASS_FWD_POOL);
    else if (pass == SB_PASS_BWD_DATA)
      r = sbh::conv_bf16c8_describe(true, d->n, d->k, d->h, d->w, d->c, buf, len);
    else
      r = sbh::conv_wgrad_c8_describe(d->n, d->c, d->h, d->w, d->k, buf, len);
    return r < 0 ? 0 : (size_t)r + 1;
  }
  switch (pass) {
    case SB_PASS_FWD:
      r = sbh::conv_igemm_describe(false, d->dtype, d->n, d->c, d->h, d->w, d->k, buf, len);
      break;
    case SB_PASS_BWD_DATA:
      r = sbh::conv_igemm_describe(true, d->dtype, d->n, d->k, d->h, d->w, d->c, buf, len);
      break;
    case SB_PASS_FWD_POOL:
      r = sbh::conv_igemm_describe(false, d->dtype, d->n, d->c, d->h, d->w, d->k, buf, len, true);
      break;
    default: r = sbh::conv_wgrad_describe(d->dtype, d->n, d->c, d->h, d->w, d->k, buf, len); break;
  }
  return r < 0 ? 0 : (size_t)r + 1;
}
