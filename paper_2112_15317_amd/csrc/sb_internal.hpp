// sb_internal.hpp -- shared device helpers and host plumbing of libsb.
// gfx950 (CDNA4) only: wave64, MFMA, 160 KB LDS per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>

#include "../../include/sb.h"

namespace sb {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16;

constexpr int kWave = 64;

// D(16x16) += A(16x4) * B(4x16), fp32 in / fp32 accumulate.
// Lane l supplies A[l%16][l/16] and B[l/16][l%16]; it receives
// D[4*(l/16)+i][l%16] in element i.
__device__ __forceinline__ f4 mfma16x16x4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// bf16 <-> fp32.  bf16 is the upper half of an fp32 bit pattern; the
// conversion to bf16 rounds to nearest, ties to even (NaN kept quiet), in
// one hardware conversion (v_cvt_pk_bf16_f32, two values per instruction).
__device__ __forceinline__ float bf16_to_f32(u16 v) {
  return __uint_as_float(((uint32_t)v) << 16);
}
__device__ __forceinline__ u16 f32_to_bf16(float f) {
  return __builtin_bit_cast(u16, (__bf16)f);
}
// lo in bits 0..15, hi in bits 16..31.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// Activation / filter element access: float (SB_F32) or bfloat16 bits held
// in u16 (SB_BF16).  Loads widen exactly to fp32; stores round to nearest.
// load4/store4 move 4 consecutive elements (16 or 8 bytes, aligned).
template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static __forceinline__ float load(const float* p, size_t i) { return p[i]; }
  __device__ static __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
  __device__ static __forceinline__ f4 load4(const float* p) {
    return *reinterpret_cast<const f4*>(p);
  }
  __device__ static __forceinline__ void store4(float* p, f4 v) { *reinterpret_cast<f4*>(p) = v; }
};
template <> struct Elem<u16> {
  __device__ static __forceinline__ float load(const u16* p, size_t i) { return bf16_to_f32(p[i]); }
  __device__ static __forceinline__ void store(u16* p, size_t i, float v) { p[i] = f32_to_bf16(v); }
  __device__ static __forceinline__ f4 load4(const u16* p) {
    uint2 u = *reinterpret_cast<const uint2*>(p);
    return f4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
              __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
  }
  __device__ static __forceinline__ void store4(u16* p, f4 v) {
    uint2 u;
    u.x = f32x2_to_bf16x2(v[0], v[1]);
    u.y = f32x2_to_bf16x2(v[2], v[3]);
    *reinterpret_cast<uint2*>(p) = u;
  }
};

// Raw buffer loads.  A 128-bit resource covers [base, base + bytes); a load at
// a byte offset outside that range returns 0 (the hardware range check).
// Staging loops select the offset (kOOB for a padded or ragged element)
// instead of selecting the loaded value, so nothing waits on the load until
// the value is stored to LDS, and the load latency hides behind the MFMAs.
// The ranges a kernel builds stay below 2^31 bytes (checked on the host).
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;
constexpr uint32_t kRsrcWord3 = 0x00020000u;   // raw, 32-bit data format (gfx9 family)

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           (int)kRsrcWord3);
}

template <typename T> struct BufLoad;
template <> struct BufLoad<float> {
  __device__ static __forceinline__ float one(rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
  }
  __device__ static __forceinline__ f4 four(rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
  }
};
template <> struct BufLoad<u16> {
  __device__ static __forceinline__ float one(rsrc_t r, uint32_t off) {
    return bf16_to_f32((u16)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0));
  }
  __device__ static __forceinline__ f4 four(rsrc_t r, uint32_t off) {
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    u2 u = __builtin_bit_cast(u2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
    return f4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
              __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
  }
};

// V consecutive bf16 in V/2 dwords (V >= 2); element 2j in the low half of
// dword j.
template <int V> struct Vec { uint32_t d[V / 2]; };

template <int V>
__device__ __forceinline__ Vec<V> load_vec(rsrc_t r, uint32_t off) {
  Vec<V> v;
  if constexpr (V == 8) {
    typedef uint32_t u4 __attribute__((ext_vector_type(4)));
    u4 t = __builtin_bit_cast(u4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
    v.d[0] = t[0]; v.d[1] = t[1]; v.d[2] = t[2]; v.d[3] = t[3];
  } else if constexpr (V == 4) {
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    u2 t = __builtin_bit_cast(u2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
    v.d[0] = t[0]; v.d[1] = t[1];
  } else {
    v.d[0] = __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
  }
  return v;
}

// V consecutive bf16 from LDS (aligned to 2V bytes).
template <int V>
__device__ __forceinline__ Vec<V> lds_vec(const u16* p) {
  Vec<V> v;
  if constexpr (V == 8) {
    typedef uint32_t u4 __attribute__((ext_vector_type(4)));
    u4 t = *reinterpret_cast<const u4*>(p);
    v.d[0] = t[0]; v.d[1] = t[1]; v.d[2] = t[2]; v.d[3] = t[3];
  } else if constexpr (V == 4) {
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    u2 t = *reinterpret_cast<const u2*>(p);
    v.d[0] = t[0]; v.d[1] = t[1];
  } else {
    v.d[0] = *reinterpret_cast<const uint32_t*>(p);
  }
  return v;
}

template <int V>
__device__ __forceinline__ void store_vec(u16* p, const Vec<V>& v) {
  if constexpr (V == 8) {
    typedef uint32_t u4 __attribute__((ext_vector_type(4)));
    *reinterpret_cast<u4*>(p) = u4{v.d[0], v.d[1], v.d[2], v.d[3]};
  } else if constexpr (V == 4) {
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    *reinterpret_cast<u2*>(p) = u2{v.d[0], v.d[1]};
  } else {
    *reinterpret_cast<uint32_t*>(p) = v.d[0];
  }
}

__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }
__host__ __device__ constexpr size_t round_up(size_t a, size_t b) { return (a + b - 1) / b * b; }

// Deterministic sum of split-reduction partials: out[i] = sum_s
// part[s*stride + i] (i < count) in a fixed order.  A block owns 64
// consecutive outputs; its four waves each sum every fourth split (s = wave,
// wave+4, ...) with several loads in flight, then wave 0 adds the four wave
// sums in order.
struct SplitSum {
  const float* part;
  int splits;
  size_t stride, count;
  __device__ __forceinline__ float operator()(size_t i, int wave, float* lds, int lane) const {
    float v = 0.f;
    if (i < count) {
      int s = wave;
      for (; s + 12 < splits; s += 16) {
        float a = part[(size_t)s * stride + i], b = part[(size_t)(s + 4) * stride + i];
        float c = part[(size_t)(s + 8) * stride + i], d = part[(size_t)(s + 12) * stride + i];
        v += a; v += b; v += c; v += d;
      }
      for (; s < splits; s += 4) v += part[(size_t)s * stride + i];
    }
    lds[wave * 64 + lane] = v;
    __syncthreads();
    return lds[lane] + lds[64 + lane] + lds[128 + lane] + lds[192 + lane];
  }
};

// Sum over splits s0 <= s < s1 of 4 consecutive partials (16-byte aligned,
// i4 a multiple of 4): part[s*stride + i4 .. +3] in increasing s (the same
// order for every output, so the result is deterministic), with four
// splits' loads in flight at a time.
__device__ __forceinline__ f4 split_sum4(const float* __restrict__ part, int s0, int s1,
                                         size_t stride, size_t i4) {
  f4 v = f4{0.f, 0.f, 0.f, 0.f};
  int s = s0;
  for (; s + 4 <= s1; s += 4) {
    const f4 a = *reinterpret_cast<const f4*>(part + (size_t)s * stride + i4);
    const f4 b = *reinterpret_cast<const f4*>(part + (size_t)(s + 1) * stride + i4);
    const f4 c = *reinterpret_cast<const f4*>(part + (size_t)(s + 2) * stride + i4);
    const f4 d = *reinterpret_cast<const f4*>(part + (size_t)(s + 3) * stride + i4);
    v += a; v += b; v += c; v += d;
  }
  for (; s < s1; ++s) v += *reinterpret_cast<const f4*>(part + (size_t)s * stride + i4);
  return v;
}

__device__ __forceinline__ f4 split_sum4(const float* __restrict__ part, int splits,
                                         size_t stride, size_t i4) {
  return split_sum4(part, 0, splits, stride, i4);
}

// Waves per block for a 4-wide split reduction of `count` outputs: 1 while
// one lane per 4 outputs already makes about 64K lanes; otherwise up to 16
// waves share out the splits (at least 4 splits a wave), so a small output
// with many splits does not leave a few hundred lanes each walking a long
// chain of dependent loads.
inline int split_waves(size_t count, int splits) {
  const size_t lanes = (count + 3) / 4;
  int g = 1;
  while (g < 16 && lanes * g < 65536 && splits >= 8 * g) g *= 2;
  return g;
}

}  // namespace sb

// Host-side helpers shared by the entry points.
namespace sbh {

inline hipStream_t stream_of(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  if (!a || !b || !abytes || !bbytes) return false;
  uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + bbytes && b0 < a0 + abytes;
}

inline sb_status launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? SB_OK : SB_ERR_HIP;
}

inline size_t dsize(int dtype) { return dtype == SB_BF16 ? 2 : 4; }

}  // namespace sbh
