// train.hip -- the loss on the complete model output and the SGD update
// (sec. 3.1 Layer Partitioning: a shard layer before the LOG_SOFTMAX layer
// gives every worker the full output, evaluated as for a complete local
// model; sec. 3.1 Modulo Layer: FC gradients are divided by K; sec. 4: SGD
// on mini-batches).
//
// log_softmax_nll_kernel: one wave per row of logits.  The lanes stride the
// row (classes c = lane, lane + 64, ...), so a row of any width costs
// ceil(classes / 64) loads per lane.  The row maximum and the sum of
// exp(z - max) are butterfly reductions over the 64 lanes (a fixed order:
// results are bitwise reproducible).  The label is compared with class
// indices and never used as an address, so an out-of-range label cannot
// reach outside the row; it yields a NaN loss and a NaN gradient row.
//
// sgd_update_kernel: a batch of tensors in one launch (as the filter packing
// does): blocks of tensor t are block0[t] .. block0[t+1]-1, each thread
// updates 4 consecutive elements with 16-byte loads and stores when the
// tensor allows it.  Pure HBM stream: 12 bytes per element.
#include "sb_internal.hpp"

#include <cmath>

namespace sb {

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ __launch_bounds__(256) void log_softmax_nll_kernel(int m, int C, int ldz,
                                                              const float* __restrict__ z,
                                                              const int* __restrict__ labels,
                                                              float scale, float* __restrict__ logp,
                                                              float* __restrict__ loss,
                                                              float* __restrict__ dz) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= m) return;                      // whole waves leave together
  const float* zr = z + (size_t)row * ldz;
  float mx = -INFINITY;
  for (int c = lane; c < C; c += 64) mx = fmaxf(mx, zr[c]);
  mx = wave_max(mx);
  float s = 0.f;
  for (int c = lane; c < C; c += 64) s += expf(zr[c] - mx);
  s = wave_sum(s);
  const float lse = mx + logf(s);
  const int lab = labels[row];
  const bool valid = lab >= 0 && lab < C;
  float picked = 0.f;                        // -logp at the label (one lane)
  for (int c = lane; c < C; c += 64) {
    const float lp = zr[c] - lse;
    if (c == lab) picked = -lp;
    if (logp) logp[(size_t)row * ldz + c] = lp;
    if (dz) {
      const float p = expf(lp);
      dz[(size_t)row * ldz + c] = valid ? scale * (p - (c == lab ? 1.f : 0.f)) : NAN;
    }
  }
  picked = wave_sum(picked);                 // exactly one nonzero term when valid
  if (loss && lane == 0) loss[row] = valid ? picked : NAN;
}

struct SgdBatch {
  float* w[SB_SGD_MAX_TENSORS];
  const float* g[SB_SGD_MAX_TENSORS];
  size_t n[SB_SGD_MAX_TENSORS];
  float step[SB_SGD_MAX_TENSORS];            // lr * scale[t]
  int vec[SB_SGD_MAX_TENSORS];               // 16-byte moves allowed
  int block0[SB_SGD_MAX_TENSORS + 1];
  int count;
};

__global__ __launch_bounds__(256) void sgd_update_kernel(SgdBatch b) {
  const int blk = blockIdx.x;
  int t = 0;
  while (t + 1 < b.count && b.block0[t + 1] <= blk) ++t;
  const size_t i = ((size_t)(blk - b.block0[t]) * 256 + threadIdx.x) * 4;
  const size_t n = b.n[t];
  if (i >= n) return;
  float* w = b.w[t];
  const float* g = b.g[t];
  const float a = -b.step[t];
  if (b.vec[t] && i + 4 <= n) {
    f4 wv = *reinterpret_cast<const f4*>(w + i);
    const f4 gv = *reinterpret_cast<const f4*>(g + i);
#pragma unroll
    for (int j = 0; j < 4; ++j) wv[j] = fmaf(a, gv[j], wv[j]);
    *reinterpret_cast<f4*>(w + i) = wv;
  } else {
    for (size_t j = i; j < i + 4 && j < n; ++j) w[j] = fmaf(a, g[j], w[j]);
  }
}

}  // namespace sb

extern "C" sb_status sb_log_softmax_nll(int m, int classes, int ldz, const float* z,
                                        const int32_t* labels, float scale, float* logp,
                                        float* loss, float* dz, void* stream) {
  if (m < 0 || classes < 1 || ldz < classes || !z || (m > 0 && !labels))
    return SB_ERR_INVALID_ARG;
  if (!std::isfinite(scale)) return SB_ERR_INVALID_ARG;
  if (m == 0) return SB_OK;
  if ((uint64_t)m * (uint64_t)ldz >= (1ull << 40)) return SB_ERR_UNSUPPORTED;
  const size_t zb = ((size_t)(m - 1) * ldz + classes) * sizeof(float);
  const size_t lb = (size_t)m * sizeof(int32_t), rb = (size_t)m * sizeof(float);
  const void* outs[3] = {logp, loss, dz};
  const size_t ob[3] = {zb, rb, zb};
  for (int i = 0; i < 3; ++i) {
    if (!outs[i]) continue;
    if (sbh::overlaps(outs[i], ob[i], z, zb) || sbh::overlaps(outs[i], ob[i], labels, lb))
      return SB_ERR_INVALID_ARG;
    for (int j = 0; j < i; ++j)
      if (outs[j] && sbh::overlaps(outs[i], ob[i], outs[j], ob[j])) return SB_ERR_INVALID_ARG;
  }
  sb::log_softmax_nll_kernel<<<(unsigned)((m + 3) / 4), 256, 0, sbh::stream_of(stream)>>>(
      m, classes, ldz, z, labels, scale, logp, loss, dz);
  return sbh::launch_status();
}

extern "C" sb_status sb_sgd_update(int count, float* const* w, const float* const* g,
                                   const size_t* n, const float* scale, float lr,
                                   void* stream) {
  if (count < 1 || count > SB_SGD_MAX_TENSORS || !w || !g || !n || !scale)
    return SB_ERR_INVALID_ARG;
  if (!std::isfinite(lr)) return SB_ERR_INVALID_ARG;
  sb::SgdBatch b{};
  b.count = count;
  long blocks = 0;
  for (int t = 0; t < count; ++t) {
    b.block0[t] = (int)blocks;
    b.w[t] = w[t];
    b.g[t] = g[t];
    b.n[t] = n[t];
    b.step[t] = (float)((double)lr * (double)scale[t]);
    if (!std::isfinite(scale[t]) || !std::isfinite(b.step[t])) return SB_ERR_INVALID_ARG;
    if (n[t] == 0) continue;
    if (!w[t] || !g[t] || n[t] >= (1ull << 40)) return SB_ERR_INVALID_ARG;
    const size_t bytes = n[t] * sizeof(float);
    for (int u = 0; u < count; ++u) {
      if (n[u] == 0) continue;
      const size_t ub = n[u] * sizeof(float);
      if (sbh::overlaps(g[t], bytes, w[u], ub)) return SB_ERR_INVALID_ARG;
      if (u < t && sbh::overlaps(w[t], bytes, w[u], ub)) return SB_ERR_INVALID_ARG;
    }
    b.vec[t] = (((uintptr_t)w[t] | (uintptr_t)g[t]) & 15) == 0;
    blocks += (long)((n[t] + 1023) / 1024);
    if (blocks >= (1l << 31)) return SB_ERR_UNSUPPORTED;
  }
  b.block0[count] = (int)blocks;
  if (blocks == 0) return SB_OK;
  sb::sgd_update_kernel<<<(unsigned)blocks, 256, 0, sbh::stream_of(stream)>>>(b);
  return sbh::launch_status();
}
