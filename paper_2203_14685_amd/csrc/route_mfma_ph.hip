// Phased matrix-core route kernel: the bf16 logit projection x.W of Eq. 1 with
// softmax and expert selection (Sec. 3.1 top-k / kTop1) for W too large to sit
// in registers (up to E = 128 experts, d a multiple of 512).
//
// Persistent blocks of 8 waves, one per CU.  A block takes two wave blocks (128
// tokens) at a time; wave w owns one 16-token tile.  W^T is staged into LDS in
// K phases of KP columns (about 128 KB: KP = 65536 / E), transposed on the way
// in 4 x 8 blocks, so W is read from L2 once per 128 tokens and there are two
// block synchronisations per phase only.  Inside a phase every wave streams its
// tile of x in 512-column chunks, one chunk ahead (16 KB per wave in flight:
// a read stream needs many bytes outstanding per CU), and runs
// v_mfma_f32_16x16x32_bf16 on B fragments read from LDS (K step ks of chunk c
// covers columns [c + 32ks, c + 32ks + 32), lane group g the 8 at c + 32ks + 8g,
// so the 4 lanes of a row load 64 contiguous bytes per instruction).  The logits
// (+ bias) then overwrite the W^T buffer and 4 lanes per token select.
#include "select.hpp"

namespace hetumoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kPhWaves = 8;
constexpr int kPhThreads = kPhWaves * kWave;
constexpr int kPhChunk = 512;             // columns per streamed chunk (16 KB per wave in flight)
constexpr int kPhLdsBytes = 65536 * 2 + 8 * 2 * 128 + 256;  // W^T phase buffer (+ row pads)

// 4 x 8 -> 8 x 4 transpose of bf16: in[j] holds row j (8 half-words); out[i]
// receives column i (4 half-words in two 32-bit words).
__device__ __forceinline__ void transpose4x8_b16(const u32x4 (&in)[4], uint2 (&out)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t a0 = in[0][i / 2], a1 = in[1][i / 2], a2 = in[2][i / 2], a3 = in[3][i / 2];
    if (i & 1) out[i] = uint2{(a0 >> 16) | (a1 & 0xffff0000u), (a2 >> 16) | (a3 & 0xffff0000u)};
    else out[i] = uint2{(a0 & 0xffffu) | (a1 << 16), (a2 & 0xffffu) | (a3 << 16)};
  }
}

template <int NT, int KMAX, bool KTOP1>
__global__ __launch_bounds__(kPhThreads) void route_mfma_ph_kernel(RouteArgs a) {
  constexpr int E = NT * 16;
  constexpr int KP = 65536 / E;        // columns per phase (a multiple of 512)
  constexpr int LDW = KP + 8;          // padded LDS row of W^T (bf16 elements)
  constexpr int KSTEPS = kPhChunk / 32;  // MFMA K steps per chunk
  constexpr int kStage = (KP / 4) * (E / 8) / kPhThreads;  // staging blocks per thread and phase
  static_assert(kStage * kPhThreads == (KP / 4) * (E / 8), "whole staging rounds");
  static_assert(E * LDW * 2 <= kPhLdsBytes, "phase buffer");
  static_assert(E * LDW * 2 >= 2 * kWave * (E + 1) * 4, "logits reuse the phase buffer");
  __shared__ __align__(16) unsigned char lds_raw[kPhLdsBytes];
  __shared__ int hist_lds[2 * 8 * E];  // [wave block of the pair][k][E]
  uint16_t* wsT = reinterpret_cast<uint16_t*>(lds_raw);
  float* lg = reinterpret_cast<float*>(lds_raw);  // [128][E + 1] after the K loop

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = lane_id();
  const int g = lane / 16, m = lane % 16;
  const int d = a.d;
  const int nchunks = d / kPhChunk;
  constexpr int CPP = KP / kPhChunk;   // chunks per phase
  const int nb = a.nb;
  const uint16_t* wg = reinterpret_cast<const uint16_t*>(a.wg);
  const uint16_t* x = reinterpret_cast<const uint16_t*>(a.x);
  const u32x4 zero = {0u, 0u, 0u, 0u};

  const int my_wbs = (nb - static_cast<int>(blockIdx.x) + static_cast<int>(gridDim.x) - 1) / static_cast<int>(gridDim.x);
  for (int pair = 0; 2 * pair < my_wbs; ++pair) {
    // wave blocks of this round: wbA (waves 0-3) and wbB (waves 4-7, may not exist)
    const int64_t wbA = blockIdx.x + static_cast<int64_t>(2 * pair) * gridDim.x;
    const bool hasB = 2 * pair + 1 < my_wbs;
    const int64_t wbB = wbA + gridDim.x;
    const int64_t my_wb = (w < 4) ? wbA : wbB;
    const bool tile_live = (w < 4) || hasB;
    const int64_t arow = my_wb * kWave + (w % 4) * 16 + m;
    const bool arow_ok = tile_live && arow < a.S;
    const u32x4* xa = reinterpret_cast<const u32x4*>(x + arow * d + 8 * g);  // + 32 ks per K step

    f32x4 acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    u32x4 xcur[KSTEPS], xnxt[KSTEPS];
#pragma unroll
    for (int v = 0; v < KSTEPS; ++v) xcur[v] = arow_ok ? xa[4 * v] : zero;

    for (int c = 0; c < nchunks; ++c) {
      if (c % CPP == 0) {
        // stage W^T[:, kp0 : kp0 + kp) of this phase
        const int kp0 = c * kPhChunk;
        const int kp = min(KP, d - kp0);
        __syncthreads();  // previous phase's fragments (or logits) consumed
        // 4 x 8 blocks (4 columns of 8 experts), kStage per thread; all loads
        // are issued before the first transpose (one L2 round trip per phase),
        // blocks past a short last phase load block 0 and store nothing
        const int nblk = (kp / 4) * (E / 8);
        u32x4 rows[kStage][4];
#pragma unroll
        for (int it = 0; it < kStage; ++it) {
          const int b = tid + it * kPhThreads;
          const int bb = b < nblk ? b : 0;
          const int kb = (bb / (E / 8)) * 4, eb = (bb % (E / 8)) * 8;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            rows[it][j] = *reinterpret_cast<const u32x4*>(wg + static_cast<int64_t>(kp0 + kb + j) * E + eb);
        }
#pragma unroll
        for (int it = 0; it < kStage; ++it) {
          const int b = tid + it * kPhThreads;
          if (b < nblk) {
            const int kb = (b / (E / 8)) * 4, eb = (b % (E / 8)) * 8;
            uint2 cols[8];
            transpose4x8_b16(rows[it], cols);
#pragma unroll
            for (int i = 0; i < 8; ++i) *reinterpret_cast<uint2*>(&wsT[(eb + i) * LDW + kb]) = cols[i];
          }
        }
        __syncthreads();
      }
      const bool more = c + 1 < nchunks;
#pragma unroll
      for (int v = 0; v < KSTEPS; ++v)
        xnxt[v] = (arow_ok && more) ? xa[(c + 1) * (kPhChunk / 8) + 4 * v] : zero;
      const int kk0 = (c % CPP) * kPhChunk + 8 * g;  // column of this lane group inside the phase
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        const bf16x8 av = __builtin_bit_cast(bf16x8, xcur[ks]);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const u32x4 braw = *reinterpret_cast<const u32x4*>(&wsT[(nt * 16 + m) * LDW + kk0 + 32 * ks]);
          acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, braw), acc[nt], 0, 0, 0);
        }
      }
#pragma unroll
      for (int v = 0; v < KSTEPS; ++v) xcur[v] = xnxt[v];
    }

    // logits (+ bias) of the 128 tokens into LDS, reusing the W^T buffer
    __syncthreads();
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int e = nt * 16 + m;
      const float bias = a.bias ? a.bias[e] : 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) lg[(w * 16 + 4 * g + i) * (E + 1) + e] = acc[nt][i] + bias;
    }
    for (int i = tid; i < 2 * a.k * E; i += kPhThreads) hist_lds[i] = 0;
    __syncthreads();
    if (a.logits && (reinterpret_cast<uintptr_t>(a.logits) & 15) == 0) {
      // 16-byte streaming stores, 4 logits of one token each (E is a multiple of 16)
      for (int o = tid; o < 2 * kWave * (E / 4); o += kPhThreads) {
        const int r = o / (E / 4), e = (o % (E / 4)) * 4;
        const int64_t s = ((r < kWave) ? wbA : wbB) * kWave + (r % kWave);
        const float* src = &lg[r * (E + 1) + e];
        if ((r < kWave || hasB) && s < a.S)
          __builtin_nontemporal_store(f32x4{src[0], src[1], src[2], src[3]}, reinterpret_cast<f32x4*>(a.logits + s * E + e));
      }
    } else if (a.logits) {  // a caller's buffer with 4-byte alignment only
      for (int o = tid; o < 2 * kWave * E; o += kPhThreads) {
        const int r = o / E, e = o % E;
        const int64_t s = ((r < kWave) ? wbA : wbB) * kWave + (r % kWave);
        if ((r < kWave || hasB) && s < a.S) a.logits[s * E + e] = lg[r * (E + 1) + e];
      }
    }
    {
      const int tt = tid / 4, j = tid % 4;  // 128 tokens, 4 lanes each
      const int half = tt / kWave;
      const int64_t s = ((half == 0) ? wbA : wbB) * kWave + (tt % kWave);
      const bool valid = (half == 0 || hasB) && s < a.S;
      select_token<4, KMAX, KTOP1>(&lg[tt * (E + 1)], E, a.k, a.normalize, j, valid, a.ids + s * a.k,
                                   a.weights + s * a.k, hist_lds + half * a.k * E);
    }
    __syncthreads();
    for (int i = tid; i < 2 * a.k * E; i += kPhThreads) {
      const int half = i / (a.k * E), rem = i % (a.k * E);
      const int r = rem / E, e = rem % E;
      if (half == 0 || hasB)
        a.hist[(static_cast<int64_t>(r) * E + e) * nb + (half == 0 ? wbA : wbB)] = hist_lds[i];
    }
  }
}

// ---------------------------------------------------------------- launch
template <int NT, int KMAX, bool KTOP1>
static hipError_t launch_ph_t(const RouteArgs& a, int grid, hipStream_t st) {
  route_mfma_ph_kernel<NT, KMAX, KTOP1><<<dim3(grid), dim3(kPhThreads), 0, st>>>(a);
  return hipGetLastError();
}

template <int NT>
static hipError_t launch_ph_nt(const RouteArgs& a, int grid, hipStream_t st) {
  if (a.kind == 1) return launch_ph_t<NT, 1, true>(a, grid, st);
  if (a.k == 1) return launch_ph_t<NT, 1, false>(a, grid, st);
  if (a.k == 2) return launch_ph_t<NT, 2, false>(a, grid, st);
  return launch_ph_t<NT, 8, false>(a, grid, st);
}

bool route_uses_mfma_ph(const RouteArgs& a) {
  if (a.kind == 2 || a.logits_in || a.dtype != 1) return false;
  if (a.E != 16 && a.E != 32 && a.E != 64 && a.E != 128) return false;
  if (a.d <= 0 || a.d % kPhChunk != 0) return false;
  return (reinterpret_cast<uintptr_t>(a.x) % 16) == 0 && (reinterpret_cast<uintptr_t>(a.wg) % 16) == 0;
}

hipError_t launch_route_mfma_ph(const RouteArgs& a, int cus, hipStream_t st) {
  // one block per CU, each taking wave blocks in pairs
  const int pairs = (a.nb + 1) / 2;
  const int grid = pairs < cus ? pairs : cus;
  switch (a.E) {
    case 16: return launch_ph_nt<1>(a, grid, st);
    case 32: return launch_ph_nt<2>(a, grid, st);
    case 64: return launch_ph_nt<4>(a, grid, st);
    case 128: return launch_ph_nt<8>(a, grid, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hetumoe
