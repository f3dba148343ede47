// api.hip -- the convolution entry points of libsb: argument validation,
// workspace sizing and dispatch to the kernels.  Nothing is enqueued unless
// every check passes.
#include "sb_internal.hpp"

namespace sbh {
size_t conv_igemm_ws(int dtype, int N, int Cin, int H, int W, int Cout);
sb_status conv_igemm(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout,
                     const void* in, const void* wt, const float* bias, const void* mask,
                     void* out, void* ws, size_t ws_bytes, int relu, hipStream_t st);
size_t conv_wgrad_ws(int dtype, int N, int C, int H, int W, int K);
int conv_igemm_describe(bool dgrad, int dtype, int N, int Cin, int H, int W, int Cout, char* buf,
                        size_t len);
int conv_wgrad_describe(int dtype, int N, int C, int H, int W, int K, char* buf, size_t len);
sb_status conv_wgrad(int dtype, int N, int C, int H, int W, int K, const void* x, const void* dy,
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
  if (d->flags & ~SB_FUSE_RELU) return SB_ERR_INVALID_ARG;
  if (pass != SB_PASS_FWD && d->flags) return SB_ERR_INVALID_ARG;
  // Kernels index weights and activations with 32-bit ints.
  if ((int64_t)d->k * d->c * 9 >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  if ((int64_t)d->n * d->c * d->h * d->w >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  if ((int64_t)d->n * d->k * d->h * d->w >= (1ll << 31)) return SB_ERR_UNSUPPORTED;
  return SB_OK;
}

extern "C" size_t sb_conv3x3_workspace_bytes(const sb_conv3x3_desc* d, int pass) {
  if (pass < SB_PASS_FWD || pass > SB_PASS_BWD_WEIGHT) return (size_t)-1;
  if (conv_check(d, pass) != SB_OK) return (size_t)-1;
  switch (pass) {
    case SB_PASS_FWD: return sbh::conv_igemm_ws(d->dtype, d->n, d->c, d->h, d->w, d->k);
    case SB_PASS_BWD_DATA: return sbh::conv_igemm_ws(d->dtype, d->n, d->k, d->h, d->w, d->c);
    default: return sbh::conv_wgrad_ws(d->dtype, d->n, d->c, d->h, d->w, d->k);
  }
}

static size_t act_bytes(const sb_conv3x3_desc* d, int ch) {
  return (size_t)d->n * ch * d->h * d->w * sbh::dsize(d->dtype);
}

extern "C" sb_status sb_conv3x3_fwd(const sb_conv3x3_desc* d, const void* x, const void* w,
                                    const float* bias, void* y, void* ws, size_t ws_bytes,
                                    void* stream) {
  sb_status s = conv_check(d, SB_PASS_FWD);
  if (s != SB_OK) return s;
  if (!x || !w || !y) return SB_ERR_INVALID_ARG;
  size_t yb = act_bytes(d, d->k), xb = act_bytes(d, d->c);
  size_t wb = (size_t)d->k * d->c * 9 * sbh::dsize(d->dtype);
  if (sbh::overlaps(y, yb, x, xb) || sbh::overlaps(y, yb, w, wb) ||
      sbh::overlaps(y, yb, bias, bias ? d->k * sizeof(float) : 0))
    return SB_ERR_INVALID_ARG;
  size_t need = sbh::conv_igemm_ws(d->dtype, d->n, d->c, d->h, d->w, d->k);
  if (need && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  if (need && (sbh::overlaps(ws, need, x, xb) || sbh::overlaps(ws, need, y, yb) ||
               sbh::overlaps(ws, need, w, wb) ||
               sbh::overlaps(ws, need, bias, bias ? d->k * sizeof(float) : 0)))
    return SB_ERR_INVALID_ARG;
  return sbh::conv_igemm(false, d->dtype, d->n, d->c, d->h, d->w, d->k, x, w, bias, nullptr, y,
                         ws, ws_bytes, (d->flags & SB_FUSE_RELU) ? 1 : 0,
                         sbh::stream_of(stream));
}

extern "C" sb_status sb_conv3x3_bwd_data(const sb_conv3x3_desc* d, const void* dy, const void* w,
                                         const void* mask, void* dx, void* ws, size_t ws_bytes,
                                         void* stream) {
  sb_status s = conv_check(d, SB_PASS_BWD_DATA);
  if (s != SB_OK) return s;
  if (!dy || !w || !dx) return SB_ERR_INVALID_ARG;
  size_t dxb = act_bytes(d, d->c), dyb = act_bytes(d, d->k);
  size_t wb = (size_t)d->k * d->c * 9 * sbh::dsize(d->dtype);
  if (sbh::overlaps(dx, dxb, dy, dyb) || sbh::overlaps(dx, dxb, w, wb) ||
      sbh::overlaps(dx, dxb, mask, mask ? dxb : 0))
    return SB_ERR_INVALID_ARG;
  size_t need = sbh::conv_igemm_ws(d->dtype, d->n, d->k, d->h, d->w, d->c);
  if (need && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  if (need && (sbh::overlaps(ws, need, dy, dyb) || sbh::overlaps(ws, need, dx, dxb) ||
               sbh::overlaps(ws, need, w, wb) ||
               sbh::overlaps(ws, need, mask, mask ? dxb : 0)))
    return SB_ERR_INVALID_ARG;
  return sbh::conv_igemm(true, d->dtype, d->n, d->k, d->h, d->w, d->c, dy, w, nullptr, mask, dx,
                         ws, ws_bytes, 0, sbh::stream_of(stream));
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
  size_t need = sbh::conv_wgrad_ws(d->dtype, d->n, d->c, d->h, d->w, d->k);
  if (need && (!ws || ws_bytes < need)) return SB_ERR_WORKSPACE;
  if (need && (sbh::overlaps(ws, need, dw, dwb) || sbh::overlaps(ws, need, db, dbb) ||
               sbh::overlaps(ws, need, x, xb) || sbh::overlaps(ws, need, dy, dyb)))
    return SB_ERR_INVALID_ARG;
  return sbh::conv_wgrad(d->dtype, d->n, d->c, d->h, d->w, d->k, x, dy, dw, db, ws, ws_bytes,
                         sbh::stream_of(stream));
}

extern "C" size_t sb_conv3x3_plan_string(const sb_conv3x3_desc* d, int pass, char* buf,
                                         size_t len) {
  if (pass < SB_PASS_FWD || pass > SB_PASS_BWD_WEIGHT) return 0;
  if (conv_check(d, pass) != SB_OK) return 0;
  int r;
  switch (pass) {
    case SB_PASS_FWD:
      r = sbh::conv_igemm_describe(false, d->dtype, d->n, d->c, d->h, d->w, d->k, buf, len);
      break;
    case SB_PASS_BWD_DATA:
      r = sbh::conv_igemm_describe(true, d->dtype, d->n, d->k, d->h, d->w, d->c, buf, len);
      break;
    default: r = sbh::conv_wgrad_describe(d->dtype, d->n, d->c, d->h, d->w, d->k, buf, len); break;
  }
  return r < 0 ? 0 : (size_t)r + 1;
}
