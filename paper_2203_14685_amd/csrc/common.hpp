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

// Value of lane (lane ^ M) for M = 1, 2, 4, 8, 16 or 32, bit for bit what a
// shuffle gives, without a trip through the LDS crossbar: M = 1 and 2
// are DPP quad permutations, M = 8 the DPP rotation of each 16-lane row by 8,
// M = 4 two DPP row shifts, each writing half of the lanes, M = 16 and 32 the
// gfx950 permlane swaps (each lane gets back its own value and its partner's:
// the one that differs from its own is the partner's, and if neither differs
// the two are equal).
template <int M>
__device__ __forceinline__ int xor_partner_i(int iv) {
  if constexpr (M == 1 || M == 2 || M == 8) {
    constexpr int ctrl = M == 1 ? 0xB1 : M == 2 ? 0x4E : 0x128;
    return __builtin_amdgcn_update_dpp(iv, iv, ctrl, 0xF, 0xF, false);
  } else if constexpr (M == 4) {
    // lanes 0-3 and 8-11 of each row (DPP banks 0 and 2) read 4 lanes up
    // (row_shl:4), lanes 4-7 and 12-15 (banks 1 and 3) 4 lanes down (row_shr:4);
    // the banks a move does not write keep the other move's value
    const int up = __builtin_amdgcn_update_dpp(iv, iv, 0x104, 0xF, 0x5, false);
    return __builtin_amdgcn_update_dpp(up, iv, 0x114, 0xF, 0xA, false);
  } else if constexpr (M == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(iv, iv, false, false);
    return static_cast<int>(r[0]) == iv ? static_cast<int>(r[1]) : static_cast<int>(r[0]);
  } else {
    static_assert(M == 32, "M is a power of two up to 32");
    const auto r = __builtin_amdgcn_permlane32_swap(iv, iv, false, false);
    return static_cast<int>(r[0]) == iv ? static_cast<int>(r[1]) : static_cast<int>(r[0]);
  }
}

template <int M, class T>
__device__ __forceinline__ T xor_partner(T v) {
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, xor_partner_i<M>(__builtin_bit_cast(int, v)));
  } else {
    static_assert(sizeof(T) == 8, "32- or 64-bit values");
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = static_cast<uint32_t>(xor_partner_i<M>(static_cast<int>(u)));
    const uint32_t hi = static_cast<uint32_t>(xor_partner_i<M>(static_cast<int>(u >> 32)));
    return __builtin_bit_cast(T, (static_cast<uint64_t>(hi) << 32) | lo);
  }
}

// The same for a mask (1, 2, 4, 8, 16 or 32) known only at run time and equal on
// all lanes; a constant mask folds to its case.
template <class T>
__device__ __forceinline__ T xor_partner(T v, int mask) {
  switch (mask) {
    case 1: return xor_partner<1>(v);
    case 2: return xor_partner<2>(v);
    case 4: return xor_partner<4>(v);
    case 8: return xor_partner<8>(v);
    case 16: return xor_partner<16>(v);
    default: return xor_partner<32>(v);
  }
}

// op(v, value of lane ^ M) for a commutative `op`.
template <int M, class T, class Op>
__device__ __forceinline__ T xor_step(T v, Op op) {
  if constexpr (M == 16 || M == 32) {
    // the swap's two results are the lane's own value and its partner's
    static_assert(sizeof(T) == 4, "32-bit values");
    const int iv = __builtin_bit_cast(int, v);
    const auto r = M == 16 ? __builtin_amdgcn_permlane16_swap(iv, iv, false, false)
                           : __builtin_amdgcn_permlane32_swap(iv, iv, false, false);
    return op(__builtin_bit_cast(T, static_cast<int>(r[0])), __builtin_bit_cast(T, static_cast<int>(r[1])));
  } else {
    return op(v, xor_partner<M>(v));
  }
}

// All-reduce over aligned groups of G lanes (G a power of two up to 64): the
// butterfly steps M = 1 .. G / 2 in increasing order.  Step 4 pairs lane i with
// lane 7 - i of its 8 (the DPP half-row mirror) instead of i ^ 4: after steps 1
// and 2 every aligned group of 4 lanes holds one value, so both partners hold
// the same and the result is the shuffle butterfly's bit for bit.
template <int G, class T, class Op>
__device__ __forceinline__ T group_reduce(T v, Op op) {
  if constexpr (G >= 2) v = xor_step<1>(v, op);
  if constexpr (G >= 4) v = xor_step<2>(v, op);
  if constexpr (G >= 8) {
    const int iv = __builtin_bit_cast(int, v);
    v = op(v, __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(iv, iv, 0x141, 0xF, 0xF, false)));
  }
  if constexpr (G >= 16) v = xor_step<8>(v, op);
  if constexpr (G >= 32) v = xor_step<16>(v, op);
  if constexpr (G >= 64) v = xor_step<32>(v, op);
  return v;
}

struct OpAdd {
  template <class T>
  __device__ __forceinline__ T operator()(T a, T b) const { return a + b; }
};
struct OpMaxI {
  __device__ __forceinline__ int operator()(int a, int b) const { return a > b ? a : b; }
};
struct OpMaxF {
  __device__ __forceinline__ float operator()(float a, float b) const { return fmaxf(a, b); }
};

__device__ __forceinline__ float wave_sum(float v) { return group_reduce<kWave>(v, OpAdd()); }

}  // namespace hetumoe
