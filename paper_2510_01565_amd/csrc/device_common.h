// Device helpers for gfx950: bf16 storage conversions, wave64 reductions,
// activations and the per-element GEMM epilogue.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "dit_internal.h"

namespace dit {

// Compile-time loop: f(std::integral_constant<int, 0>) ... f(<N-1>).  Register
// arrays indexed by its counter never become dynamically indexed (which would
// move them to scratch memory).
template <class F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

typedef uint16_t bf16_t;  // raw bfloat16 storage
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(bf16_t u) { return __uint_as_float(((uint32_t)u) << 16); }

// fp32 -> bf16, round to nearest even (hardware conversion on gfx950)
__device__ __forceinline__ bf16_t f2bf(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(bf16_t, b);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f2bf(v); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// GELU, tanh form: 0.5 x (1 + tanh(u)) = x * sigmoid(2u), u = sqrt(2/pi) (x + 0.044715 x^3).
// exp2 and the reciprocal are single transcendental-unit instructions (about
// 1 ulp each); for very negative x the exponential overflows to +inf and the
// result is -0.
__device__ __forceinline__ float gelu_tanh(float x) {
  const float k = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float t = k * x * (1.0f + 0.044715f * x * x);
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(t));
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }

// Per-row facts an epilogue needs, computed once per output tile row.
struct RowEntry {
  int req;  // request index
  int pos;  // position in the padded joint layout of Q / K / V^T
  int gi;   // grid row of an image token, -1 for text
  int gj;   // grid column of an image token
};

__device__ __forceinline__ RowEntry make_row_entry(const BatchMeta& meta, int R) {
  const RowInfo ri = row_info(meta, R);
  RowEntry e;
  e.req = ri.req;
  e.pos = padded_pos(meta, ri);
  if (ri.is_img) {
    const int gw = meta.grid_w[ri.req];
    e.gi = ri.local / gw;
    e.gj = ri.local - e.gi * gw;
  } else {
    e.gi = -1;
    e.gj = 0;
  }
  return e;
}

// One output element of a GEMM epilogue.  `y` already includes the bias;
// `y_pair` is the value of the partner column n ^ 1 (RoPE pairs), bias included.
template <typename T>
__device__ __forceinline__ void epilogue_element(const EpiArgs& e, const RowEntry& row, int m, int n, float y,
                                                 float y_pair) {
  switch (e.mode) {
    case EPI_STORE_F32:
      ((float*)e.out)[(long)m * e.ldo + n] = y;
      break;
    case EPI_STORE_T:
      ((T*)e.out)[(long)m * e.ldo + n] = from_f32<T>(y);
      break;
    case EPI_GELU:
      ((T*)e.out)[(long)m * e.ldo + e.col0 + n] = from_f32<T>(gelu_tanh(y));
      break;
    case EPI_RESID: {
      const float g = e.mods[(long)row.req * e.mods_ld + e.gate_off + n];
      float* xo = (float*)e.out + (long)m * e.ldo + n;
      *xo = *xo + g * y;
      break;
    }
    case EPI_QKV: {
      if (n >= e.n_qkv) {
        ((T*)e.gelu_out)[(long)m * e.gelu_ld + e.gelu_col0 + (n - e.n_qkv)] = from_f32<T>(gelu_tanh(y));
        break;
      }
      const int H = e.hidden, d = e.head_dim;
      const int which = n / H;
      const int hn = n - which * H;
      const int h = hn / d, dd = hn - h * d;
      float v = y;
      if (which < 2 && row.gi >= 0) {
        const int half = d >> 1;
        const int pos = (dd < half) ? row.gi : row.gj;
        const int kk = (dd < half ? dd : dd - half) >> 1;
        const float2 cs = e.rope[pos * (d >> 2) + kk];
        // even: u cos - v sin ; odd: u sin + v cos  (u = even element, v = odd element)
        v = (dd & 1) ? (y_pair * cs.y + y * cs.x) : (y * cs.x - y_pair * cs.y);
      }
      if (which == 0)
        ((T*)e.q)[((long)h * e.T + row.pos) * d + dd] = from_f32<T>(v);
      else if (which == 1)
        ((T*)e.k)[((long)h * e.T + row.pos) * d + dd] = from_f32<T>(v);
      else
        ((T*)e.vt)[((long)h * d + dd) * e.vt_ld + vt_slot(row.pos)] = from_f32<T>(v);
      break;
    }
    default:
      break;
  }
}

// 16 consecutive output columns n .. n+15 (n a multiple of 16) of one row m,
// bias already added.  Vectorised form of epilogue_element: every store and
// residual update is 16 bytes wide except the transposed V^T scatter.
template <typename T>
__device__ __forceinline__ void store16(T* dst, const float* v) {
  if constexpr (sizeof(T) == 2) {
    uint4 a, b;
    a.x = pack_bf16x2(v[0], v[1]);
    a.y = pack_bf16x2(v[2], v[3]);
    a.z = pack_bf16x2(v[4], v[5]);
    a.w = pack_bf16x2(v[6], v[7]);
    b.x = pack_bf16x2(v[8], v[9]);
    b.y = pack_bf16x2(v[10], v[11]);
    b.z = pack_bf16x2(v[12], v[13]);
    b.w = pack_bf16x2(v[14], v[15]);
    ((uint4*)dst)[0] = a;
    ((uint4*)dst)[1] = b;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) ((float4*)dst)[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  }
}

template <typename T>
__device__ __forceinline__ void epilogue_segment16(const EpiArgs& e, const RowEntry& row, int m, int n, float* v) {
  switch (e.mode) {
    case EPI_STORE_F32:
      store16<float>((float*)e.out + (long)m * e.ldo + n, v);
      break;
    case EPI_STORE_T:
      store16<T>((T*)e.out + (long)m * e.ldo + n, v);
      break;
    case EPI_GELU:
#pragma unroll
      for (int q = 0; q < 16; ++q) v[q] = gelu_tanh(v[q]);
      store16<T>((T*)e.out + (long)m * e.ldo + e.col0 + n, v);
      break;
    case EPI_RESID: {
      const float4* g = (const float4*)(e.mods + (long)row.req * e.mods_ld + e.gate_off + n);
      float4* xo = (float4*)((float*)e.out + (long)m * e.ldo + n);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 gv = g[q];
        float4 xv = xo[q];
        xv.x += gv.x * v[4 * q];
        xv.y += gv.y * v[4 * q + 1];
        xv.z += gv.z * v[4 * q + 2];
        xv.w += gv.w * v[4 * q + 3];
        xo[q] = xv;
      }
      break;
    }
    case EPI_QKV: {
      if (n >= e.n_qkv) {
#pragma unroll
        for (int q = 0; q < 16; ++q) v[q] = gelu_tanh(v[q]);
        store16<T>((T*)e.gelu_out + (long)m * e.gelu_ld + e.gelu_col0 + (n - e.n_qkv), v);
        break;
      }
      const int H = e.hidden, d = e.head_dim;
      const int which = n / H;
      const int hn = n - which * H;
      const int h = hn / d, dd0 = hn - h * d;
      if (which < 2 && row.gi >= 0) {
        const int half = d >> 1;
        const int pos = (dd0 < half) ? row.gi : row.gj;
        const int k0 = (dd0 < half ? dd0 : dd0 - half) >> 1;
        const float2* cs = e.rope + pos * (d >> 2) + k0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float2 c = cs[q];
          const float u = v[2 * q], w = v[2 * q + 1];
          v[2 * q] = u * c.x - w * c.y;
          v[2 * q + 1] = u * c.y + w * c.x;
        }
      }
      if (which == 0)
        store16<T>((T*)e.q + ((long)h * e.T + row.pos) * d + dd0, v);
      else if (which == 1)
        store16<T>((T*)e.k + ((long)h * e.T + row.pos) * d + dd0, v);
      else {
        T* vt = (T*)e.vt + ((long)h * d + dd0) * e.vt_ld + vt_slot(row.pos);
#pragma unroll
        for (int q = 0; q < 16; ++q) vt[(long)q * e.vt_ld] = from_f32<T>(v[q]);
      }
      break;
    }
    default:
      break;
  }
}

// XCD-aware block remap: hardware dispatches block b to XCD b % 8; return an
// index such that every XCD owns one contiguous range of indices.
// Word 3 of a raw buffer resource on gfx9-family targets: 32-bit data format,
// so untyped dword loads are range-checked against num_records and return
// zeros past it.
constexpr int kBufferWord3 = 0x00020000;

__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int per = nblocks / 8, rem = nblocks % 8;
  const int xcd = bid % 8, idx = bid / 8;
  return (xcd < rem) ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
}

}  // namespace dit
