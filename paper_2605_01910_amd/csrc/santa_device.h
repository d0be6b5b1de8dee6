// santa_device.h -- gfx950 device helpers for the SANTA decode kernels:
// 16-byte row-chunk loads, bf16 dot products, DPP reductions within 16-lane
// rows, wave reductions and scans.  Wave size is 64 (CDNA).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "santa_plan.h"

namespace santa {

constexpr float kInf = __builtin_huge_valf();

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
typedef unsigned int nt_u32x4 __attribute__((ext_vector_type(4)));
typedef float nt_f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// a.x*b.x + a.y*b.y + c on packed bf16 pairs (v_dot2c_f32_bf16)
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// ---------------------------------------------------------------------------
// 8 consecutive features of one row, loaded with 128-bit loads.
// bf16: one dwordx4 of packed pairs; f32: two dwordx4.
// ---------------------------------------------------------------------------
template <typename E>
struct Chunk;

template <>
struct Chunk<uint16_t> {
  uint4 w;
  __device__ __forceinline__ static Chunk zero() { return Chunk{make_uint4(0, 0, 0, 0)}; }
  __device__ __forceinline__ static Chunk load(const uint16_t *p) {
    return Chunk{*reinterpret_cast<const uint4 *>(p)};
  }
  // non-temporal (nt): for rows streamed once, so they do not displace
  // reused lines in L2 and the memory-side cache
  __device__ __forceinline__ static Chunk load_nt(const uint16_t *p) {
    const nt_u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const nt_u32x4 *>(p));
    return Chunk{make_uint4(v[0], v[1], v[2], v[3])};
  }
  __device__ __forceinline__ void to_float(float (&f)[8]) const {
    f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x); f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
    f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z); f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
  }
  __device__ __forceinline__ void require() const {
    asm volatile("" ::"v"(w.x), "v"(w.y), "v"(w.z), "v"(w.w));
  }
  // <this, q> over the 8 features
  __device__ __forceinline__ float dot(const Chunk &q) const {
    float a = dot2_bf16(w.x, q.w.x, 0.0f);
    a = dot2_bf16(w.y, q.w.y, a);
    a = dot2_bf16(w.z, q.w.z, a);
    return dot2_bf16(w.w, q.w.w, a);
  }
};

template <>
struct Chunk<float> {
  float4 a, b;
  __device__ __forceinline__ static Chunk zero() {
    return Chunk{make_float4(0, 0, 0, 0), make_float4(0, 0, 0, 0)};
  }
  __device__ __forceinline__ static Chunk load(const float *p) {
    return Chunk{reinterpret_cast<const float4 *>(p)[0], reinterpret_cast<const float4 *>(p)[1]};
  }
  __device__ __forceinline__ static Chunk load_nt(const float *p) {
    const nt_f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const nt_f32x4 *>(p));
    const nt_f32x4 y = __builtin_nontemporal_load(reinterpret_cast<const nt_f32x4 *>(p) + 1);
    return Chunk{make_float4(x[0], x[1], x[2], x[3]), make_float4(y[0], y[1], y[2], y[3])};
  }
  __device__ __forceinline__ void to_float(float (&f)[8]) const {
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  __device__ __forceinline__ void require() const {
    asm volatile("" ::"v"(a.x), "v"(a.y), "v"(a.z), "v"(a.w));
    asm volatile("" ::"v"(b.x), "v"(b.y), "v"(b.z), "v"(b.w));
  }
  __device__ __forceinline__ float dot(const Chunk &q) const {
    float s = a.x * q.a.x;
    s = fmaf(a.y, q.a.y, s); s = fmaf(a.z, q.a.z, s); s = fmaf(a.w, q.a.w, s);
    s = fmaf(b.x, q.b.x, s); s = fmaf(b.y, q.b.y, s); s = fmaf(b.z, q.b.z, s);
    return fmaf(b.w, q.b.w, s);
  }
};

// 8 consecutive features of one row of an OCP FP8 E4M3 cache (one byte per
// feature), loaded with one 64-bit load.  The codes widen exactly: to float32
// with v_cvt_pk_f32_fp8 (two codes per instruction) and to packed bfloat16
// with v_cvt_scalef32_pk_bf16_fp8 at scale 1 (every E4M3 value, subnormals
// included, is a bfloat16 value).  The per-(batch, KV head) dequantisation
// scale is applied by the caller, outside the feature loops.
typedef unsigned int nt_u32x2 __attribute__((ext_vector_type(2)));

template <>
struct Chunk<uint8_t> {
  uint2 w;
  __device__ __forceinline__ static Chunk zero() { return Chunk{make_uint2(0, 0)}; }
  __device__ __forceinline__ static Chunk load(const uint8_t *p) {
    return Chunk{*reinterpret_cast<const uint2 *>(p)};
  }
  __device__ __forceinline__ static Chunk load_nt(const uint8_t *p) {
    const nt_u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const nt_u32x2 *>(p));
    return Chunk{make_uint2(v[0], v[1])};
  }
  __device__ __forceinline__ void to_float(float (&f)[8]) const {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    const f32x2_t a = __builtin_amdgcn_cvt_pk_f32_fp8(w.x, false);
    const f32x2_t b = __builtin_amdgcn_cvt_pk_f32_fp8(w.x, true);
    const f32x2_t c = __builtin_amdgcn_cvt_pk_f32_fp8(w.y, false);
    const f32x2_t d = __builtin_amdgcn_cvt_pk_f32_fp8(w.y, true);
    f[0] = a[0]; f[1] = a[1]; f[2] = b[0]; f[3] = b[1];
    f[4] = c[0]; f[5] = c[1]; f[6] = d[0]; f[7] = d[1];
  }
  __device__ __forceinline__ void require() const { asm volatile("" ::"v"(w.x), "v"(w.y)); }
  // the 8 codes as 4 packed bfloat16 pairs (features 2i, 2i+1 in word i)
  __device__ __forceinline__ uint4 to_bf16() const {
    return make_uint4(
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w.x, 1.0f, false)),
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w.x, 1.0f, true)),
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w.y, 1.0f, false)),
        __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w.y, 1.0f, true)));
  }
  // <this, q> over the 8 features with a bfloat16 query
  __device__ __forceinline__ float dot(const Chunk<uint16_t> &q) const {
    const uint4 k = to_bf16();
    float a = dot2_bf16(k.x, q.w.x, 0.0f);
    a = dot2_bf16(k.y, q.w.y, a);
    a = dot2_bf16(k.z, q.w.z, a);
    return dot2_bf16(k.w, q.w.w, a);
  }
};

// Element type of q and out for a cache of element type E: the cache's own
// type, except bfloat16 queries and outputs for an FP8 cache.
template <typename E>
struct QElemOf {
  using type = E;
};
template <>
struct QElemOf<uint8_t> {
  using type = uint16_t;
};
template <typename E>
using QE = typename QElemOf<E>::type;

// ---------------------------------------------------------------------------
// Cross-lane helpers.  DPP controls (gfx9 encoding): quad_perm [1,0,3,2] = 0xB1,
// quad_perm [2,3,0,1] = 0x4E, row_half_mirror = 0x141, row_mirror = 0x140.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xf, 0xf, false));
}

// Sum over the 16 lanes of a DPP row; every lane of the row gets the total.
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  v += dpp<0x140>(v);
  return v;
}

__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  return v;
}

// Lane-wise combination with the lane 16 (32) apart, on every lane, using the
// gfx950 lane-swap instructions (VALU, no LDS crossbar).  Both lanes of a pair
// see the operands in the same order, so they get bitwise-identical results.
__device__ __forceinline__ float xor16_sum(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float xor32_sum(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float xor16_max(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float xor32_max(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}

// Wave-wide max / sum; every lane gets the same value.
__device__ __forceinline__ float wave_max(float v) { return xor32_max(xor16_max(row16_max(v))); }
__device__ __forceinline__ float wave_sum(float v) { return xor32_sum(xor16_sum(row16_sum(v))); }

// DPP with a fill value for lanes that have no source lane.
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ float dpp_fill(float fill, float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill),
                                                               __builtin_bit_cast(int, v), CTRL,
                                                               ROWS, 0xf, false));
}

// Inclusive prefix sum over the 64 lanes in a fixed order: row_shr 1/2/4/8
// within each row of 16, then row_bcast 15 and 31 across rows.
__device__ __forceinline__ float wave_incl_scan(float v) {
  v += dpp_fill<0x111>(0.0f, v);
  v += dpp_fill<0x112>(0.0f, v);
  v += dpp_fill<0x114>(0.0f, v);
  v += dpp_fill<0x118>(0.0f, v);
  v += dpp_fill<0x142, 0xa>(0.0f, v);
  v += dpp_fill<0x143, 0xc>(0.0f, v);
  return v;
}

// Inclusive prefix max over the 64 lanes (exact).
__device__ __forceinline__ float wave_incl_max(float v) {
  const float ninf = -__builtin_huge_valf();
  v = fmaxf(v, dpp_fill<0x111>(ninf, v));
  v = fmaxf(v, dpp_fill<0x112>(ninf, v));
  v = fmaxf(v, dpp_fill<0x114>(ninf, v));
  v = fmaxf(v, dpp_fill<0x118>(ninf, v));
  v = fmaxf(v, dpp_fill<0x142, 0xa>(ninf, v));
  v = fmaxf(v, dpp_fill<0x143, 0xc>(ninf, v));
  return v;
}

// Value of the previous lane (wave_shr:1); lane 0 gets `fill`.
__device__ __forceinline__ float wave_prev(float fill, float v) { return dpp_fill<0x138>(fill, v); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------------------
// KV addressing
// ---------------------------------------------------------------------------
// Dequantisation scales of row (b, kvh) of an FP8 cache (K, V); 1 for other
// element types, whose stored values are the values.
template <typename E>
__device__ __forceinline__ float2 kv_scales(const KvView &kv, int b, int kvh, int Hkv) {
  if constexpr (sizeof(E) == 1) {
    const int64_t r = (int64_t)b * Hkv + kvh;
    return make_float2(kv.ks[r], kv.vs[r]);
  } else {
    return make_float2(1.0f, 1.0f);
  }
}
__device__ __forceinline__ int seq_len(const KvView &kv, int b) {
  if (!kv.ctx) return kv.n_k;
  int L = kv.ctx[b];
  return L < 0 ? 0 : (L > kv.n_k ? kv.n_k : L);
}

// Element offset of token `pos` of sequence b, KV head kvh (feature 0).
template <bool PAGED>
__device__ __forceinline__ int64_t row_offset(const KvView &kv, int b, int kvh, int pos) {
  if constexpr (PAGED) {
    const int page = kv.bt[(int64_t)b * kv.max_pages + (pos >> kv.ps_log2)];
    return (int64_t)page * kv.sb + (int64_t)(pos & ((1 << kv.ps_log2) - 1)) * kv.sn +
           (int64_t)kvh * kv.sh;
  } else {
    return (int64_t)b * kv.sb + (int64_t)pos * kv.sn + (int64_t)kvh * kv.sh;
  }
}

}  // namespace santa
