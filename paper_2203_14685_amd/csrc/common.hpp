// Device helpers shared by the gfx950 kernels: element types, 16-byte row
// vectors, bf16 <-> fp32 conversion and wave64 primitives.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hetumoe {

constexpr int kWave = 64;           // CDNA wavefront width
constexpr int kBlock = 256;         // default threads per block
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kTokensPerHistBlock = 64;  // capacity-scan granularity: one wave block of 64 tokens

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// bf16 storage type: the upper 16 bits of an IEEE binary32.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_lo(uint32_t packed) { return __uint_as_float(packed << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t packed) { return __uint_as_float(packed & 0xffff0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest, ties to even, by gfx950's packed conversion
// (v_cvt_pk_bf16_f32): values beyond the bf16 range become infinities and NaNs
// stay NaNs.  Checked on MI355X bit for bit against the integer rounding
// u + 0x7fff + ((u >> 16) & 1) over 33 million finite inputs (denormals, exact
// ties and the top of the range included).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) { return pack_bf16x2(f, 0.f) & 0xffffu; }

// A 16-byte chunk of a row holds 4 fp32 or 8 bf16 elements.
template <typename T> struct Chunk;
template <> struct Chunk<float> {
  static constexpr int kElems = 4;
  __device__ __forceinline__ static void unpack(const u32x4& v, float* out) {
    out[0] = __uint_as_float(v.x);
    out[1] = __uint_as_float(v.y);
    out[2] = __uint_as_float(v.z);
    out[3] = __uint_as_float(v.w);
  }
  __device__ __forceinline__ static u32x4 pack(const float* in) {
    u32x4 v;
    v.x = __float_as_uint(in[0]);
    v.y = __float_as_uint(in[1]);
    v.z = __float_as_uint(in[2]);
    v.w = __float_as_uint(in[3]);
    return v;
  }
};
template <> struct Chunk<bf16_t> {
  static constexpr int kElems = 8;
  __device__ __forceinline__ static void unpack(const u32x4& v, float* out) {
    out[0] = bf16_lo(v.x); out[1] = bf16_hi(v.x);
    out[2] = bf16_lo(v.y); out[3] = bf16_hi(v.y);
    out[4] = bf16_lo(v.z); out[5] = bf16_hi(v.z);
    out[6] = bf16_lo(v.w); out[7] = bf16_hi(v.w);
  }
  __device__ __forceinline__ static u32x4 pack(const float* in) {
    u32x4 v;
    v.x = pack_bf16x2(in[0], in[1]);
    v.y = pack_bf16x2(in[2], in[3]);
    v.z = pack_bf16x2(in[4], in[5]);
    v.w = pack_bf16x2(in[6], in[7]);
    return v;
  }
};

__device__ __forceinline__ float load_elem(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_elem(const bf16_t* p, int64_t i) {
  return __uint_as_float(static_cast<uint32_t>(p[i].bits) << 16);
}

// 8 x 8 transpose of bf16: in[j] holds row j (8 half-words, lowest first);
// out[i] receives column i.
__device__ __forceinline__ void transpose8x8_b16(const u32x4 (&in)[8], u32x4 (&out)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t wd[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t a = in[2 * q][i / 2], b = in[2 * q + 1][i / 2];
      wd[q] = (i & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
    out[i] = u32x4{wd[0], wd[1], wd[2], wd[3]};
  }
}

__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

// Number of set bits of `mask` in lanes below the calling lane.
__device__ __forceinline__ int popc_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

}  // namespace hetumoe
