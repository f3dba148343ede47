// pool.hip -- fused ReLU + 2x2/2 max pooling with window codes, and its
// backward (sec. 2.2: pooling subsamples the features between convolutional
// stages).  Both directions are pure data movement, bound by HBM bandwidth:
// each thread owns PER_THREAD horizontally adjacent windows, so it reads
// 2*PER_THREAD contiguous elements from each of two input rows and writes
// PER_THREAD outputs and codes; neighbouring threads touch neighbouring
// addresses.  No window is shared between threads, so no atomics are needed.
#include "sb_internal.hpp"

namespace sb {

// Window code: bits 0-1 = row-major position of the first maximum, bit 7 =
// maximum <= 0 (ReLU blocks the gradient).
template <typename T, int PER_THREAD>
__global__ __launch_bounds__(256) void relu_maxpool_fwd_kernel(
    const T* __restrict__ x, T* __restrict__ y, uint8_t* __restrict__ idx,
    uint32_t Wo, uint32_t groups_per_row, uint32_t total_groups) {
  uint32_t g = blockIdx.x * 256u + threadIdx.x;
  if (g >= total_groups) return;
  uint32_t row = g / groups_per_row;               // (n*C + c)*Ho + oh
  uint32_t ow0 = (g - row * groups_per_row) * PER_THREAD;
  const size_t W = 2 * (size_t)Wo;
  const T* p0 = x + (size_t)row * 2 * W + 2 * ow0;  // input rows 2*oh, 2*oh+1
  const T* p1 = p0 + W;
  size_t o = (size_t)row * Wo + ow0;
#pragma unroll
  for (int j = 0; j < PER_THREAD; ++j) {
    if (ow0 + j >= Wo) break;
    float v0 = Elem<T>::load(p0, 2 * j), v1 = Elem<T>::load(p0, 2 * j + 1);
    float v2 = Elem<T>::load(p1, 2 * j), v3 = Elem<T>::load(p1, 2 * j + 1);
    float m = v0;
    uint32_t a = 0;
    if (v1 > m) { m = v1; a = 1; }
    if (v2 > m) { m = v2; a = 2; }
    if (v3 > m) { m = v3; a = 3; }
    bool pos = m > 0.0f;
    Elem<T>::store(y, o + j, pos ? m : 0.0f);
    idx[o + j] = (uint8_t)(a | (pos ? 0u : 0x80u));
  }
}

template <typename T, int PER_THREAD>
__global__ __launch_bounds__(256) void relu_maxpool_bwd_kernel(
    const T* __restrict__ dy, const uint8_t* __restrict__ idx, T* __restrict__ dx,
    uint32_t Wo, uint32_t groups_per_row, uint32_t total_groups) {
  uint32_t g = blockIdx.x * 256u + threadIdx.x;
  if (g >= total_groups) return;
  uint32_t row = g / groups_per_row;
  uint32_t ow0 = (g - row * groups_per_row) * PER_THREAD;
  const size_t W = 2 * (size_t)Wo;
  T* p0 = dx + (size_t)row * 2 * W + 2 * ow0;
  T* p1 = p0 + W;
  size_t o = (size_t)row * Wo + ow0;
#pragma unroll
  for (int j = 0; j < PER_THREAD; ++j) {
    if (ow0 + j >= Wo) break;
    float gv = Elem<T>::load(dy, o + j);
    uint32_t code = idx[o + j];
    bool live = !(code & 0x80u);
    uint32_t a = code & 3u;
    Elem<T>::store(p0, 2 * j, (live && a == 0) ? gv : 0.0f);
    Elem<T>::store(p0, 2 * j + 1, (live && a == 1) ? gv : 0.0f);
    Elem<T>::store(p1, 2 * j, (live && a == 2) ? gv : 0.0f);
    Elem<T>::store(p1, 2 * j + 1, (live && a == 3) ? gv : 0.0f);
  }
}

// Vector form: 4 windows per thread, output width a multiple of 4 and every
// tensor 16-byte aligned.  The two input rows of the 4 windows are 8
// contiguous elements each (16 bytes in bf16, 32 in fp32), the 4 outputs and
// the 4 codes contiguous too: every access is a whole vector.
template <typename T> struct V8;                   // 8 elements
template <> struct V8<float> {
  typedef float t __attribute__((ext_vector_type(8)));
  __device__ static float get(const t& v, int i) { return v[i]; }
  __device__ static void put(t& v, int i, float x) { v[i] = x; }
};
template <> struct V8<u16> {
  typedef u16 t __attribute__((ext_vector_type(8)));
  __device__ static float get(const t& v, int i) { return bf16_to_f32(v[i]); }
  __device__ static void put(t& v, int i, float x) { v[i] = f32_to_bf16(x); }
};
template <typename T> struct V4;                   // 4 elements
template <> struct V4<float> {
  typedef float t __attribute__((ext_vector_type(4)));
  __device__ static float get(const t& v, int i) { return v[i]; }
  __device__ static void put(t& v, int i, float x) { v[i] = x; }
};
template <> struct V4<u16> {
  typedef u16 t __attribute__((ext_vector_type(4)));
  __device__ static float get(const t& v, int i) { return bf16_to_f32(v[i]); }
  __device__ static void put(t& v, int i, float x) { v[i] = f32_to_bf16(x); }
};

template <typename T>
__global__ __launch_bounds__(256) void relu_maxpool_fwd_vec(
    const T* __restrict__ x, T* __restrict__ y, uint8_t* __restrict__ idx,
    uint32_t Wo, uint32_t groups_per_row, uint32_t total_groups) {
  typedef typename V8<T>::t in_t;
  typedef typename V4<T>::t out_t;
  uint32_t g = blockIdx.x * 256u + threadIdx.x;
  if (g >= total_groups) return;
  uint32_t row = g / groups_per_row;               // (n*C + c)*Ho + oh
  uint32_t ow0 = (g - row * groups_per_row) * 4;
  const size_t W = 2 * (size_t)Wo;
  const T* p0 = x + (size_t)row * 2 * W + 2 * ow0;
  const in_t r0 = *reinterpret_cast<const in_t*>(p0);
  const in_t r1 = *reinterpret_cast<const in_t*>(p0 + W);
  out_t o;
  uint32_t codes = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float m = V8<T>::get(r0, 2 * j);
    uint32_t a = 0;
    const float v1 = V8<T>::get(r0, 2 * j + 1), v2 = V8<T>::get(r1, 2 * j),
                v3 = V8<T>::get(r1, 2 * j + 1);
    if (v1 > m) { m = v1; a = 1; }
    if (v2 > m) { m = v2; a = 2; }
    if (v3 > m) { m = v3; a = 3; }
    const bool pos = m > 0.0f;
    V4<T>::put(o, j, pos ? m : 0.0f);
    codes |= (a | (pos ? 0u : 0x80u)) << (8 * j);
  }
  const size_t oo = (size_t)row * Wo + ow0;
  *reinterpret_cast<out_t*>(y + oo) = o;
  *reinterpret_cast<uint32_t*>(idx + oo) = codes;
}

template <typename T>
__global__ __launch_bounds__(256) void relu_maxpool_bwd_vec(
    const T* __restrict__ dy, const uint8_t* __restrict__ idx, T* __restrict__ dx,
    uint32_t Wo, uint32_t groups_per_row, uint32_t total_groups) {
  typedef typename V8<T>::t row_t;
  typedef typename V4<T>::t in_t;
  uint32_t g = blockIdx.x * 256u + threadIdx.x;
  if (g >= total_groups) return;
  uint32_t row = g / groups_per_row;
  uint32_t ow0 = (g - row * groups_per_row) * 4;
  const size_t W = 2 * (size_t)Wo;
  const size_t oo = (size_t)row * Wo + ow0;
  const in_t gv = *reinterpret_cast<const in_t*>(dy + oo);
  const uint32_t codes = *reinterpret_cast<const uint32_t*>(idx + oo);
  row_t r0, r1;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t code = (codes >> (8 * j)) & 0xffu;
    const bool live = !(code & 0x80u);
    const uint32_t a = code & 3u;
    const float v = V4<T>::get(gv, j);
    V8<T>::put(r0, 2 * j, (live && a == 0) ? v : 0.0f);
    V8<T>::put(r0, 2 * j + 1, (live && a == 1) ? v : 0.0f);
    V8<T>::put(r1, 2 * j, (live && a == 2) ? v : 0.0f);
    V8<T>::put(r1, 2 * j + 1, (live && a == 3) ? v : 0.0f);
  }
  T* p0 = dx + (size_t)row * 2 * W + 2 * ow0;
  *reinterpret_cast<row_t*>(p0) = r0;
  *reinterpret_cast<row_t*>(p0 + W) = r1;
}

// Channel-blocked tensors (SB_NCHW8C): a thread owns one window of 8
// channels (one 16-byte bf16 piece per pixel): its two input rows are 16
// contiguous elements each, its output and codes 8 contiguous elements and
// bytes, and neighbouring threads take neighbouring windows.
template <typename T>
__global__ __launch_bounds__(256) void relu_maxpool_fwd_c8(
    const T* __restrict__ x, T* __restrict__ y, uint8_t* __restrict__ idx, uint32_t Wo,
    uint32_t total) {
  const uint32_t g = blockIdx.x * 256u + threadIdx.x;   // ((n*CB + cb)*Ho + oh)*Wo + ow
  if (g >= total) return;
  const uint32_t row = g / Wo, ow = g - row * Wo;
  const size_t W = 2 * (size_t)Wo;
  const T* p0 = x + ((size_t)row * 2 * W + 2 * ow) * 8;
  const T* p1 = p0 + W * 8;
  typedef typename V8<T>::t v8;
  const v8 a0 = *reinterpret_cast<const v8*>(p0), a1 = *reinterpret_cast<const v8*>(p0 + 8);
  const v8 b0 = *reinterpret_cast<const v8*>(p1), b1 = *reinterpret_cast<const v8*>(p1 + 8);
  v8 o;
  uint32_t codes[2] = {0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float m = V8<T>::get(a0, e);
    uint32_t c = 0;
    const float v1 = V8<T>::get(a1, e), v2 = V8<T>::get(b0, e), v3 = V8<T>::get(b1, e);
    if (v1 > m) { m = v1; c = 1; }
    if (v2 > m) { m = v2; c = 2; }
    if (v3 > m) { m = v3; c = 3; }
    const bool pos = m > 0.0f;
    V8<T>::put(o, e, pos ? m : 0.0f);
    codes[e / 4] |= (c | (pos ? 0u : 0x80u)) << (8 * (e % 4));
  }
  *reinterpret_cast<v8*>(y + (size_t)g * 8) = o;
  *reinterpret_cast<uint2*>(idx + (size_t)g * 8) = make_uint2(codes[0], codes[1]);
}

template <typename T>
__global__ __launch_bounds__(256) void relu_maxpool_bwd_c8(
    const T* __restrict__ dy, const uint8_t* __restrict__ idx, T* __restrict__ dx, uint32_t Wo,
    uint32_t total) {
  const uint32_t g = blockIdx.x * 256u + threadIdx.x;
  if (g >= total) return;
  const uint32_t row = g / Wo, ow = g - row * Wo;
  const size_t W = 2 * (size_t)Wo;
  typedef typename V8<T>::t v8;
  const v8 gv = *reinterpret_cast<const v8*>(dy + (size_t)g * 8);
  const uint2 cw = *reinterpret_cast<const uint2*>(idx + (size_t)g * 8);
  v8 a0, a1, b0, b1;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t code = ((e < 4 ? cw.x : cw.y) >> (8 * (e % 4))) & 0xffu;
    const bool live = !(code & 0x80u);
    const uint32_t c = code & 3u;
    const float v = V8<T>::get(gv, e);
    V8<T>::put(a0, e, (live && c == 0) ? v : 0.0f);
    V8<T>::put(a1, e, (live && c == 1) ? v : 0.0f);
    V8<T>::put(b0, e, (live && c == 2) ? v : 0.0f);
    V8<T>::put(b1, e, (live && c == 3) ? v : 0.0f);
  }
  T* p0 = dx + ((size_t)row * 2 * W + 2 * ow) * 8;
  T* p1 = p0 + W * 8;
  *reinterpret_cast<v8*>(p0) = a0;
  *reinterpret_cast<v8*>(p0 + 8) = a1;
  *reinterpret_cast<v8*>(p1) = b0;
  *reinterpret_cast<v8*>(p1 + 8) = b1;
}

template <typename T>
static sb_status pool_launch_c8(bool fwd, int n, int c, int h, int w, const void* in,
                                const uint8_t* idx_in, void* out, uint8_t* idx_out,
                                hipStream_t st) {
  const uint32_t Wo = (uint32_t)(w / 2);
  const uint32_t total = (uint32_t)n * (c / 8) * (h / 2) * Wo;
  dim3 grid((total + 255) / 256), block(256);
  if (fwd)
    relu_maxpool_fwd_c8<T><<<grid, block, 0, st>>>((const T*)in, (T*)out, idx_out, Wo, total);
  else
    relu_maxpool_bwd_c8<T><<<grid, block, 0, st>>>((const T*)in, idx_in, (T*)out, Wo, total);
  return sbh::launch_status();
}

template <typename T>
static sb_status pool_launch(bool fwd, int n, int c, int h, int w, const void* in,
                             const uint8_t* idx_in, void* out, uint8_t* idx_out,
                             hipStream_t st) {
  uint32_t Wo = (uint32_t)(w / 2);
  uint32_t rows = (uint32_t)n * c * (h / 2);
  const uintptr_t al = (uintptr_t)in | (uintptr_t)idx_in | (uintptr_t)out | (uintptr_t)idx_out;
  if (Wo % 4 == 0 && al % 16 == 0) {
    const uint32_t gpr = Wo / 4, total = rows * gpr;
    dim3 grid((total + 255) / 256), block(256);
    if (fwd)
      relu_maxpool_fwd_vec<T><<<grid, block, 0, st>>>((const T*)in, (T*)out, idx_out, Wo, gpr,
                                                      total);
    else
      relu_maxpool_bwd_vec<T><<<grid, block, 0, st>>>((const T*)in, idx_in, (T*)out, Wo, gpr,
                                                      total);
    return sbh::launch_status();
  }
  constexpr int PT = 2;
  uint32_t gpr = (Wo + PT - 1) / PT;
  uint32_t total = rows * gpr;
  dim3 grid((total + 255) / 256), block(256);
  if (fwd)
    relu_maxpool_fwd_kernel<T, PT><<<grid, block, 0, st>>>(
        (const T*)in, (T*)out, idx_out, Wo, gpr, total);
  else
    relu_maxpool_bwd_kernel<T, PT><<<grid, block, 0, st>>>(
        (const T*)in, idx_in, (T*)out, Wo, gpr, total);
  return sbh::launch_status();
}

}  // namespace sb

using namespace sb;

static sb_status pool_check(int n, int c, int h, int w, int dtype, int layout) {
  if (n <= 0 || c <= 0 || h <= 0 || w <= 0) return SB_ERR_INVALID_ARG;
  if ((h & 1) || (w & 1)) return SB_ERR_INVALID_ARG;
  if (dtype != SB_F32 && dtype != SB_BF16) return SB_ERR_INVALID_ARG;
  if (layout != SB_NCHW && layout != SB_NCHW8C) return SB_ERR_INVALID_ARG;
  if (layout == SB_NCHW8C && c % 8) return SB_ERR_INVALID_ARG;
  // 32-bit window indexing inside the kernels.
  if ((uint64_t)n * c * h * w >= (1ull << 32)) return SB_ERR_UNSUPPORTED;
  return SB_OK;
}

extern "C" sb_status sb_relu_maxpool_fwd(int n, int c, int h, int w, int dtype, int layout,
                                         const void* x, void* y, uint8_t* idx,
                                         void* stream) {
  sb_status s = pool_check(n, c, h, w, dtype, layout);
  if (s != SB_OK) return s;
  if (!x || !y || !idx) return SB_ERR_INVALID_ARG;
  size_t es = sbh::dsize(dtype);
  size_t in_b = (size_t)n * c * h * w * es, out_n = (size_t)n * c * (h / 2) * (w / 2);
  if (sbh::overlaps(x, in_b, y, out_n * es) || sbh::overlaps(x, in_b, idx, out_n) ||
      sbh::overlaps(y, out_n * es, idx, out_n))
    return SB_ERR_INVALID_ARG;
  hipStream_t st = sbh::stream_of(stream);
  if (layout == SB_NCHW8C) {
    // 16-byte pieces (8 bf16 or 2 x 4 fp32), 8-byte code groups.
    if (((uintptr_t)x | (uintptr_t)y) & 15 || (uintptr_t)idx & 7) return SB_ERR_INVALID_ARG;
    return dtype == SB_F32 ? pool_launch_c8<float>(true, n, c, h, w, x, nullptr, y, idx, st)
                           : pool_launch_c8<u16>(true, n, c, h, w, x, nullptr, y, idx, st);
  }
  return dtype == SB_F32 ? pool_launch<float>(true, n, c, h, w, x, nullptr, y, idx, st)
                         : pool_launch<u16>(true, n, c, h, w, x, nullptr, y, idx, st);
}

extern "C" sb_status sb_relu_maxpool_bwd(int n, int c, int h, int w, int dtype, int layout,
                                         const void* dy, const uint8_t* idx, void* dx,
                                         void* stream) {
  sb_status s = pool_check(n, c, h, w, dtype, layout);
  if (s != SB_OK) return s;
  if (!dy || !idx || !dx) return SB_ERR_INVALID_ARG;
  size_t es = sbh::dsize(dtype);
  size_t out_b = (size_t)n * c * h * w * es, in_n = (size_t)n * c * (h / 2) * (w / 2);
  if (sbh::overlaps(dx, out_b, dy, in_n * es) || sbh::overlaps(dx, out_b, idx, in_n))
    return SB_ERR_INVALID_ARG;
  hipStream_t st = sbh::stream_of(stream);
  if (layout == SB_NCHW8C) {
    if (((uintptr_t)dy | (uintptr_t)dx) & 15 || (uintptr_t)idx & 7) return SB_ERR_INVALID_ARG;
    return dtype == SB_F32 ? pool_launch_c8<float>(false, n, c, h, w, dy, idx, dx, nullptr, st)
                           : pool_launch_c8<u16>(false, n, c, h, w, dy, idx, dx, nullptr, st);
  }
  return dtype == SB_F32 ? pool_launch<float>(false, n, c, h, w, dy, idx, dx, nullptr, st)
                         : pool_launch<u16>(false, n, c, h, w, dy, idx, dx, nullptr, st);
}
