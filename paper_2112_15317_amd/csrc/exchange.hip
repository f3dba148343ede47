// exchange.hip -- data movement of the modulo and shard layers around the FC
// shards when the buffers of every emulated worker sit on this device
// (sec. 3.1, Modulo Layer and Shard Layer; sec. 3.2, Group MP Extension).
//
// Worker w's slot starts w * stride elements from a base pointer.  Workers
// form MP groups of mp consecutive ids; a call serves one group (first id
// g):
//   modulo fwd, iteration k:  gathered[b]  = local[g + b/s][k*s + b%s]
//   modulo bwd, iteration k:  dlocal[g + b/s][k*s + b%s] = sum_w dgathered[g + w][b]
//   shard fwd:                full[m][r*Ns + c] = parts[g + r][m][c]
//   shard bwd:                dparts[g + r][m][c] = sum_w dfull[g + w][m][r*Ns + c]
// (s = B / mp; sums over w = 0 .. mp-1 in that order.)
//
// All four are pure HBM streams: every output element is written once and
// every input element the group owns is read once.  One thread moves V = 4
// consecutive fp32 elements (16-byte loads and stores) when every row and
// slot keeps 16-byte alignment, else one; the index arithmetic per element
// group is a few integer divisions, far below the memory time.
#include "sb_internal.hpp"

namespace sb {

template <int V> struct VecOf;
template <> struct VecOf<4> { using T = f4; };
template <> struct VecOf<1> { using T = float; };

template <int V>
__device__ __forceinline__ typename VecOf<V>::T ld(const float* p) {
  return *reinterpret_cast<const typename VecOf<V>::T*>(p);
}
template <int V>
__device__ __forceinline__ void st(float* p, typename VecOf<V>::T v) {
  *reinterpret_cast<typename VecOf<V>::T*>(p) = v;
}

// One thread per V consecutive features of one gathered example.
template <int V>
__global__ __launch_bounds__(256) void modulo_fwd_kernel(const float* __restrict__ local,
                                                         size_t ls, float* __restrict__ out,
                                                         int g, int k, int s, int F,
                                                         size_t groups) {
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= groups) return;
  const size_t e = q * V;
  const int b = (int)(e / F), f = (int)(e - (size_t)b * F);
  const float* src = local + (size_t)(g + b / s) * ls + (size_t)(k * s + b % s) * F + f;
  st<V>(out + e, ld<V>(src));
}

template <int V>
__global__ __launch_bounds__(256) void modulo_bwd_kernel(const float* __restrict__ dg,
                                                         size_t dgs, float* __restrict__ dl,
                                                         size_t dls, int g, int mp, int k, int s,
                                                         int F, size_t groups) {
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= groups) return;
  const size_t e = q * V;
  const int b = (int)(e / F), f = (int)(e - (size_t)b * F);
  const float* src = dg + (size_t)g * dgs + e;
  typename VecOf<V>::T acc = ld<V>(src);
  for (int w = 1; w < mp; ++w) acc += ld<V>(src + (size_t)w * dgs);
  st<V>(dl + (size_t)(g + b / s) * dls + (size_t)(k * s + b % s) * F + f, acc);
}

// One thread per V consecutive columns of one row of the full input.
template <int V>
__global__ __launch_bounds__(256) void shard_fwd_kernel(const float* __restrict__ parts,
                                                        size_t ps, float* __restrict__ full,
                                                        int g, int mp, int Ns, size_t groups) {
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= groups) return;
  const size_t e = q * V, width = (size_t)mp * Ns;
  const size_t m = e / width;
  const int col = (int)(e - m * width), r = col / Ns, c = col - r * Ns;
  st<V>(full + e, ld<V>(parts + (size_t)(g + r) * ps + m * Ns + c));
}

// One thread per V consecutive columns of one row of one worker's slice;
// outputs ordered (worker r, row m, column c).
template <int V>
__global__ __launch_bounds__(256) void shard_bwd_kernel(const float* __restrict__ dfull,
                                                        size_t dfs, float* __restrict__ dparts,
                                                        size_t dps, int g, int mp, int M, int Ns,
                                                        size_t groups) {
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= groups) return;
  const size_t e = q * V, slice = (size_t)M * Ns;
  const int r = (int)(e / slice);
  const size_t rem = e - (size_t)r * slice;
  const size_t m = rem / Ns;
  const int c = (int)(rem - m * Ns);
  const float* src = dfull + (size_t)g * dfs + m * ((size_t)mp * Ns) + (size_t)r * Ns + c;
  typename VecOf<V>::T acc = ld<V>(src);
  for (int w = 1; w < mp; ++w) acc += ld<V>(src + (size_t)w * dfs);
  st<V>(dparts + (size_t)(g + r) * dps + rem, acc);
}

// Model averaging: one thread per V consecutive elements of one averaging
// set (shard r): the set's slots r, mp + r, ... are read in increasing
// worker id and all of them receive the sum divided by their count.
template <int V>
__global__ __launch_bounds__(256) void model_average_kernel(float* __restrict__ p, size_t stride,
                                                            int mp, int groups, size_t per_slot,
                                                            size_t total) {
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= total) return;
  const int r = (int)(q / per_slot);
  float* base = p + (size_t)r * stride + (q - (size_t)r * per_slot) * V;
  const size_t step = (size_t)mp * stride;
  typename VecOf<V>::T acc = ld<V>(base);
  for (int g = 1; g < groups; ++g) acc += ld<V>(base + g * step);
  const float cnt = (float)groups;
  if constexpr (V == 1) {
    acc = acc / cnt;
  } else {
#pragma unroll
    for (int j = 0; j < V; ++j) acc[j] = acc[j] / cnt;
  }
  for (int g = 0; g < groups; ++g) st<V>(base + g * step, acc);
}

// Model averaging of replicas held in separate buffers: the n elements of
// every replica are replaced by their mean (sum in increasing replica id,
// one division).  The replica pointers travel in the kernel arguments.
struct ReplicaSet {
  float* p[SB_MAX_REPLICAS];
};

template <int V>
__global__ __launch_bounds__(256) void replica_average_kernel(ReplicaSet rs, int replicas,
                                                              size_t total) {
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= total) return;
  const size_t e = q * V;
  typename VecOf<V>::T acc = ld<V>(rs.p[0] + e);
  for (int g = 1; g < replicas; ++g) acc += ld<V>(rs.p[g] + e);
  const float cnt = (float)replicas;
  if constexpr (V == 1) {
    acc = acc / cnt;
  } else {
#pragma unroll
    for (int j = 0; j < V; ++j) acc[j] = acc[j] / cnt;
  }
  for (int g = 0; g < replicas; ++g) st<V>(rs.p[g] + e, acc);
}

}  // namespace sb

using namespace sb;

namespace {

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// Byte range of the group's slots [g, g + mp) of a slotted buffer.
size_t group_bytes(size_t stride, int mp, size_t slot) {
  return ((size_t)(mp - 1) * stride + slot) * sizeof(float);
}

bool group_ok(int workers, int mp, int iproc) {
  return mp >= 1 && workers >= mp && workers % mp == 0 && iproc >= 0 && iproc < workers;
}

unsigned blocks_for(size_t groups) { return (unsigned)((groups + 255) / 256); }

bool modulo_ok(const sb_modulo_desc* d, int iproc, int k) {
  return d && group_ok(d->workers, d->mp, iproc) && d->batch >= d->mp && d->batch % d->mp == 0 &&
         d->features >= 1 && k >= 0 && k < d->mp &&
         (uint64_t)d->batch * (uint64_t)d->features < (1ull << 40);
}

bool shard_ok(const sb_shard_desc* d, int iproc) {
  return d && group_ok(d->workers, d->mp, iproc) && d->rows >= 1 && d->shard >= 1 &&
         (uint64_t)d->rows * (uint64_t)d->shard * (uint64_t)d->mp < (1ull << 40);
}

}  // namespace

extern "C" sb_status sb_modulo_fwd(const sb_modulo_desc* d, int iproc, int k, const float* local,
                                   size_t local_stride, float* gathered, void* stream) {
  if (!modulo_ok(d, iproc, k) || !local || !gathered) return SB_ERR_INVALID_ARG;
  const size_t slot = (size_t)d->batch * d->features;
  if (local_stride < slot) return SB_ERR_INVALID_ARG;
  const int mp = d->mp, g = (iproc / mp) * mp, s = d->batch / mp;
  const float* lg = local + (size_t)g * local_stride;
  if (sbh::overlaps(gathered, slot * sizeof(float), lg, group_bytes(local_stride, mp, slot)))
    return SB_ERR_INVALID_ARG;
  hipStream_t st = sbh::stream_of(stream);
  const bool v4 = d->features % 4 == 0 && local_stride % 4 == 0 && aligned16(local) &&
                  aligned16(gathered);
  if (v4)
    modulo_fwd_kernel<4><<<blocks_for(slot / 4), 256, 0, st>>>(local, local_stride, gathered, g,
                                                               k, s, d->features, slot / 4);
  else
    modulo_fwd_kernel<1><<<blocks_for(slot), 256, 0, st>>>(local, local_stride, gathered, g, k,
                                                           s, d->features, slot);
  return sbh::launch_status();
}

extern "C" sb_status sb_modulo_bwd(const sb_modulo_desc* d, int iproc, int k,
                                   const float* dgathered, size_t dg_stride, float* dlocal,
                                   size_t dl_stride, void* stream) {
  if (!modulo_ok(d, iproc, k) || !dgathered || !dlocal) return SB_ERR_INVALID_ARG;
  const size_t slot = (size_t)d->batch * d->features;
  if (dg_stride < slot || dl_stride < slot) return SB_ERR_INVALID_ARG;
  const int mp = d->mp, g = (iproc / mp) * mp, s = d->batch / mp;
  if (sbh::overlaps(dlocal + (size_t)g * dl_stride, group_bytes(dl_stride, mp, slot),
                    dgathered + (size_t)g * dg_stride, group_bytes(dg_stride, mp, slot)))
    return SB_ERR_INVALID_ARG;
  hipStream_t st = sbh::stream_of(stream);
  const bool v4 = d->features % 4 == 0 && dg_stride % 4 == 0 && dl_stride % 4 == 0 &&
                  aligned16(dgathered) && aligned16(dlocal);
  if (v4)
    modulo_bwd_kernel<4><<<blocks_for(slot / 4), 256, 0, st>>>(
        dgathered, dg_stride, dlocal, dl_stride, g, mp, k, s, d->features, slot / 4);
  else
    modulo_bwd_kernel<1><<<blocks_for(slot), 256, 0, st>>>(
        dgathered, dg_stride, dlocal, dl_stride, g, mp, k, s, d->features, slot);
  return sbh::launch_status();
}

extern "C" sb_status sb_shard_fwd(const sb_shard_desc* d, int iproc, const float* parts,
                                  size_t parts_stride, float* full, void* stream) {
  if (!shard_ok(d, iproc) || !parts || !full) return SB_ERR_INVALID_ARG;
  const size_t slot = (size_t)d->rows * d->shard;
  if (parts_stride < slot) return SB_ERR_INVALID_ARG;
  const int mp = d->mp, g = (iproc / mp) * mp;
  const size_t total = slot * mp;
  if (sbh::overlaps(full, total * sizeof(float), parts + (size_t)g * parts_stride,
                    group_bytes(parts_stride, mp, slot)))
    return SB_ERR_INVALID_ARG;
  hipStream_t st = sbh::stream_of(stream);
  const bool v4 = d->shard % 4 == 0 && parts_stride % 4 == 0 && aligned16(parts) &&
                  aligned16(full);
  if (v4)
    shard_fwd_kernel<4><<<blocks_for(total / 4), 256, 0, st>>>(parts, parts_stride, full, g, mp,
                                                               d->shard, total / 4);
  else
    shard_fwd_kernel<1><<<blocks_for(total), 256, 0, st>>>(parts, parts_stride, full, g, mp,
                                                           d->shard, total);
  return sbh::launch_status();
}

extern "C" sb_status sb_shard_bwd(const sb_shard_desc* d, int iproc, const float* dfull,
                                  size_t df_stride, float* dparts, size_t dp_stride,
                                  void* stream) {
  if (!shard_ok(d, iproc) || !dfull || !dparts) return SB_ERR_INVALID_ARG;
  const size_t slot = (size_t)d->rows * d->shard;
  const int mp = d->mp, g = (iproc / mp) * mp;
  const size_t fslot = slot * mp;
  if (df_stride < fslot || dp_stride < slot) return SB_ERR_INVALID_ARG;
  if (sbh::overlaps(dparts + (size_t)g * dp_stride, group_bytes(dp_stride, mp, slot),
                    dfull + (size_t)g * df_stride, group_bytes(df_stride, mp, fslot)))
    return SB_ERR_INVALID_ARG;
  hipStream_t st = sbh::stream_of(stream);
  const bool v4 = d->shard % 4 == 0 && df_stride % 4 == 0 && dp_stride % 4 == 0 &&
                  aligned16(dfull) && aligned16(dparts);
  const size_t total = fslot;   // outputs: mp slices of [M][Ns]
  if (v4)
    shard_bwd_kernel<4><<<blocks_for(total / 4), 256, 0, st>>>(
        dfull, df_stride, dparts, dp_stride, g, mp, d->rows, d->shard, total / 4);
  else
    shard_bwd_kernel<1><<<blocks_for(total), 256, 0, st>>>(
        dfull, df_stride, dparts, dp_stride, g, mp, d->rows, d->shard, total);
  return sbh::launch_status();
}

extern "C" sb_status sb_model_average(int workers, int mp, size_t n, float* params, size_t stride,
                                      void* stream) {
  if (workers < 1 || mp < 1 || workers % mp != 0) return SB_ERR_INVALID_ARG;
  if (n == 0) return SB_OK;
  if (!params || stride < n) return SB_ERR_INVALID_ARG;
  if ((uint64_t)(workers - 1) * stride + n >= (1ull << 40)) return SB_ERR_UNSUPPORTED;
  const int groups = workers / mp;
  if (groups == 1) return SB_OK;                  // one worker per set: nothing to average
  hipStream_t st = sbh::stream_of(stream);
  const bool v4 = n % 4 == 0 && stride % 4 == 0 && aligned16(params);
  if (v4) {
    const size_t per = n / 4, total = per * mp;
    model_average_kernel<4><<<blocks_for(total), 256, 0, st>>>(params, stride, mp, groups, per,
                                                               total);
  } else {
    const size_t total = n * mp;
    model_average_kernel<1><<<blocks_for(total), 256, 0, st>>>(params, stride, mp, groups, n,
                                                               total);
  }
  return sbh::launch_status();
}

extern "C" sb_status sb_model_average_replicas(int replicas, size_t n, float* const* params,
                                               void* stream) {
  if (replicas < 1 || replicas > SB_MAX_REPLICAS || !params) return SB_ERR_INVALID_ARG;
  for (int g = 0; g < replicas; ++g)
    if (!params[g]) return SB_ERR_INVALID_ARG;
  if (n == 0) return SB_OK;
  if (n >= (1ull << 40)) return SB_ERR_UNSUPPORTED;
  const size_t bytes = n * sizeof(float);
  for (int g = 0; g < replicas; ++g)
    for (int h = g + 1; h < replicas; ++h)
      if (sbh::overlaps(params[g], bytes, params[h], bytes)) return SB_ERR_INVALID_ARG;
  if (replicas == 1) return SB_OK;                // one replica: already its own mean
  ReplicaSet rs{};
  bool v4 = n % 4 == 0;
  for (int g = 0; g < replicas; ++g) {
    rs.p[g] = params[g];
    v4 = v4 && aligned16(params[g]);
  }
  hipStream_t st = sbh::stream_of(stream);
  if (v4)
    replica_average_kernel<4><<<blocks_for(n / 4), 256, 0, st>>>(rs, replicas, n / 4);
  else
    replica_average_kernel<1><<<blocks_for(n), 256, 0, st>>>(rs, replicas, n);
  return sbh::launch_status();
}
