// Device-side helpers shared by the gfx950 kernels of the resident-expert layer.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <algorithm>

typedef __bf16 bf16_t;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2_t;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4_t;
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short s16x8_t;
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

#define DEVI __device__ __forceinline__

DEVI float to_f32(float v) { return v; }
DEVI float to_f32(bf16_t v) { return (float)v; }

template <class T> DEVI T from_f32(float v);
template <> DEVI float from_f32<float>(float v) { return v; }
// fptrunc f32 -> bf16 rounds to nearest even (v_cvt_pk_bf16_f32 on gfx950)
template <> DEVI bf16_t from_f32<bf16_t>(float v) { return (bf16_t)v; }

// Number of elements of T in one 16-byte vector.
template <class T> struct Vec16 { static constexpr int N = 16 / sizeof(T); };

// Load / store 16 bytes of T as fp32 values.
DEVI void load16_f32(const float* p, float* out) {
  f32x4_t v = *reinterpret_cast<const f32x4_t*>(p);
  out[0] = v[0]; out[1] = v[1]; out[2] = v[2]; out[3] = v[3];
}
DEVI void load16_f32(const bf16_t* p, float* out) {
  bf16x8_t v = *reinterpret_cast<const bf16x8_t*>(p);
#pragma unroll
  for (int i = 0; i < 8; ++i) out[i] = (float)v[i];
}
DEVI void store16_f32(float* p, const float* in) {
  f32x4_t v = {in[0], in[1], in[2], in[3]};
  *reinterpret_cast<f32x4_t*>(p) = v;
}
DEVI void store16_f32(bf16_t* p, const float* in) {
  bf16x8_t v;
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (bf16_t)in[i];
  *reinterpret_cast<bf16x8_t*>(p) = v;
}

DEVI float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

DEVI float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

DEVI float silu_f(float g) { return g / (1.0f + expf(-g)); }
DEVI float sigmoid_f(float g) { return 1.0f / (1.0f + expf(-g)); }

// MFMA 32x32x16 operand fragment (lane l: index l%32 of the M or N side,
// k = 8*(l/32) + 0..7) read with two ds_read_b64_tr_b16 from an LDS array
// whose rows are k and whose columns are M/N (row stride `stride` bytes):
// in each 16-lane group, lane 4r+q addresses 4 consecutive columns of row r
// and receives, transposed, one column of the group's 4x16 block.
DEVI bf16x8_t frag_tr(const char* base, int stride, int row0, int col0) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, i = lane & 15;
  const int col = col0 + 16 * (g & 1) + 4 * (i & 3);
  s16x4_t v[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int row = row0 + 8 * (g >> 1) + 4 * h + (i >> 2);
    v[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_s16x4_t*)(base + (size_t)row * stride + col * 2));
  }
  const s16x8_t both = __builtin_shufflevector(v[0], v[1], 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8_t, both);
}

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
