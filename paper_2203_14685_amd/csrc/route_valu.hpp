// Route kernel on the vector ALUs: the logit projection x.W of Eq. 1 (any
// dtype and shape), softmax and expert selection, one thread per token.
// Instantiated per element type in route_valu_f32.hip and route_valu_bf16.hip.
#pragma once

#include "select.hpp"

namespace hetumoe {

// ---------------------------------------------------------------- VALU route
// One thread per token, one wave (64 tokens) per block.  Logits for EC experts
// at a time are accumulated in registers from the token's row of x and a
// [kDJ, EC] tile of W staged in LDS.
constexpr int kDJ = 64;

template <typename T, int EC, int KMAX, bool KTOP1>
__global__ __launch_bounds__(kWave) void route_valu_kernel(RouteArgs a) {
  extern __shared__ int hist_lds[];  // [E]
  __shared__ float wg_s[kDJ][EC];

  const int tid = threadIdx.x;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kWave + tid;
  const bool valid = s < a.S;
  const int E = a.E, k = a.k;

  TopkState<KMAX> tk;
  tk.init();
  Ktop1State kt;
  kt.init(E / k);
  int32_t* my_ids = a.ids + s * k;
  float* my_w = a.weights + s * k;

  const T* xrow = reinterpret_cast<const T*>(a.x) + s * a.d;
  constexpr int kEl = Chunk<T>::kElems;

  for (int e0 = 0; e0 < E; e0 += EC) {
    float acc[EC];
#pragma unroll
    for (int i = 0; i < EC; ++i) acc[i] = 0.f;

    if (a.logits_in) {
      if (valid) {
#pragma unroll
        for (int i = 0; i < EC; ++i)
          if (e0 + i < E) acc[i] = a.logits[s * E + e0 + i];
      }
    } else {
      const T* wg = reinterpret_cast<const T*>(a.wg);
      for (int j0 = 0; j0 < a.d; j0 += kDJ) {
        __syncthreads();  // previous tile fully consumed
        for (int t = tid; t < kDJ * EC; t += kWave) {
          const int jj = t / EC, ii = t % EC;
          const int j = j0 + jj, e = e0 + ii;
          wg_s[jj][ii] = (j < a.d && e < E) ? load_elem(wg, static_cast<int64_t>(j) * E + e) : 0.f;
        }
        __syncthreads();
        if (valid) {
          const int jend = min(kDJ, a.d - j0);
          const u32x4* xv = reinterpret_cast<const u32x4*>(xrow + j0);
          if (jend == kDJ) {
            // full chunk: issue all of its loads before the first FMA
            constexpr int kNC = kDJ / kEl;
            u32x4 xc[kNC];
#pragma unroll
            for (int c = 0; c < kNC; ++c) xc[c] = xv[c];
#pragma unroll
            for (int c = 0; c < kNC; ++c) {
              float xe[kEl];
              Chunk<T>::unpack(xc[c], xe);
#pragma unroll
              for (int q = 0; q < kEl; ++q) {
                const float* wrow = wg_s[c * kEl + q];
#pragma unroll
                for (int i = 0; i < EC; ++i) acc[i] = fmaf(xe[q], wrow[i], acc[i]);
              }
            }
          } else {
            for (int c = 0; c < jend / kEl; ++c) {
              float xe[kEl];
              Chunk<T>::unpack(xv[c], xe);
#pragma unroll
              for (int q = 0; q < kEl; ++q) {
                const float* wrow = wg_s[c * kEl + q];
#pragma unroll
                for (int i = 0; i < EC; ++i) acc[i] = fmaf(xe[q], wrow[i], acc[i]);
              }
            }
          }
        }
      }
      if (valid) {
#pragma unroll
        for (int i = 0; i < EC; ++i) {
          if (e0 + i < E) {
            if (a.bias) acc[i] += a.bias[e0 + i];
            if (a.logits) a.logits[s * E + e0 + i] = acc[i];
          }
        }
      }
    }

    if (valid) {
#pragma unroll
      for (int i = 0; i < EC; ++i) {
        if (e0 + i < E) {
          if constexpr (KTOP1) kt.push(acc[i], e0 + i, my_ids, my_w);
          else tk.push(acc[i], e0 + i);
        }
      }
    }
  }
  if constexpr (!KTOP1) {
    if (valid) tk.finish(k, a.normalize, my_ids, my_w);
  }
  wave_block_hist(hist_lds, true, s, valid, blockIdx.x, a);
}

// ---------------------------------------------------------------- split VALU route
// P = 8 lanes per token (E a power of two, 8 <= E <= 64), one block per wave
// block of 64 tokens.  Lane j of a token takes 16-byte chunks j, j + P, ... of
// the token's row, so the P lanes read P x 16 contiguous bytes per load and a
// lane keeps kSplitU loads in flight.  W is staged in LDS as fp32 in phases of
// KC rows.  The E partial sums are then reduced over the P lanes by recursive
// halving: at each step a lane keeps one half of its remaining sums (the upper
// half where its lane bit is set), adds the partner's copy of that half and
// hands over the other, which leaves each lane E / P finished logits.
constexpr int kSplitP = 8;
constexpr int kSplitU = 8;             // chunks in flight per lane
constexpr int kSplitWFloats = 8192;    // 32 KB of W per phase

template <int H>
__device__ __forceinline__ void halve_sums(float* v, int msk, bool upper) {
#pragma unroll
  for (int i = 0; i < H; ++i) {
    const float give = upper ? v[i] : v[i + H];
    const float keep = upper ? v[i + H] : v[i];
    v[i] = keep + __shfl_xor(give, msk);
  }
}

template <typename T, int E, int KMAX, bool KTOP1>
__global__ __launch_bounds__(kWave * kSplitP) void route_valu_split_kernel(RouteArgs a) {
  constexpr int P = kSplitP;
  constexpr int kThreads = kWave * P;
  constexpr int kEl = Chunk<T>::kElems;
  constexpr int KC = kSplitWFloats / E;  // W rows per phase (a multiple of kEl)
  constexpr int NV = E / P;              // finished logits per lane
  static_assert(E >= P && (E & (E - 1)) == 0 && KC % kEl == 0, "split route shape");
  extern __shared__ int hist_lds[];      // [k][E]
  __shared__ __align__(16) float ws[KC * E];
  __shared__ float lg[kWave * (E + 1)];

  const int tid = threadIdx.x;
  const int tok = tid / P, j = tid % P;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kWave + tok;
  const bool valid = s < a.S;
  const T* wg = reinterpret_cast<const T*>(a.wg);
  const u32x4* xv = reinterpret_cast<const u32x4*>(reinterpret_cast<const T*>(a.x) + (valid ? s : 0) * a.d);
  const u32x4 zero = {0u, 0u, 0u, 0u};

  float acc[E];
#pragma unroll
  for (int i = 0; i < E; ++i) acc[i] = 0.f;

  for (int k0 = 0; k0 < a.d; k0 += KC) {
    const int kc = min(KC, a.d - k0);  // a multiple of kEl (d is)
    const int nch = kc / kEl, cbase = k0 / kEl;
    // the phase's first loads of x go out before W is staged
    u32x4 xc[kSplitU];
#pragma unroll
    for (int u = 0; u < kSplitU; ++u) {
      const int c = u * P + j;
      xc[u] = (valid && c < nch) ? xv[cbase + c] : zero;
    }
    if (k0 > 0) __syncthreads();       // previous phase consumed
    const u32x4* wv = reinterpret_cast<const u32x4*>(wg + static_cast<int64_t>(k0) * E);
    for (int t = tid; t < kc * E / kEl; t += kThreads) {
      float f[kEl];
      Chunk<T>::unpack(wv[t], f);
#pragma unroll
      for (int q = 0; q < kEl; ++q) ws[t * kEl + q] = f[q];
    }
    __syncthreads();
    for (int c0 = 0; c0 < nch; c0 += P * kSplitU) {
      if (c0 > 0) {
#pragma unroll
        for (int u = 0; u < kSplitU; ++u) {
          const int c = c0 + u * P + j;
          xc[u] = (valid && c < nch) ? xv[cbase + c] : zero;
        }
      }
#pragma unroll
      for (int u = 0; u < kSplitU; ++u) {
        const int c = c0 + u * P + j;
        if (c < nch) {
          float xe[kEl];
          Chunk<T>::unpack(xc[u], xe);
#pragma unroll
          for (int q = 0; q < kEl; ++q) {
            const float* wr = &ws[(c * kEl + q) * E];
#pragma unroll
            for (int i = 0; i < E; ++i) acc[i] = fmaf(xe[q], wr[i], acc[i]);
          }
        }
      }
    }
  }

  // reduce over the P lanes of the token: lane j ends with experts [off, off + NV)
  halve_sums<E / 2>(acc, 1, j & 1);
  halve_sums<E / 4>(acc, 2, j & 2);
  halve_sums<E / 8>(acc, 4, j & 4);
  const int off = ((j & 1) ? E / 2 : 0) + ((j & 2) ? E / 4 : 0) + ((j & 4) ? E / 8 : 0);

  for (int i = tid; i < a.k * E; i += kThreads) hist_lds[i] = 0;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int e = off + i;
    const float v = acc[i] + (a.bias ? a.bias[e] : 0.f);
    lg[tok * (E + 1) + e] = v;
    if (a.logits && valid) a.logits[s * E + e] = v;
  }
  __syncthreads();
  select_token<P, KMAX, KTOP1>(&lg[tok * (E + 1)], E, a.k, a.normalize, j, valid, a.ids + s * a.k,
                               a.weights + s * a.k, hist_lds);
  __syncthreads();
  for (int i = tid; i < a.k * E; i += kThreads)
    a.hist[static_cast<int64_t>(i) * a.nb + blockIdx.x] = hist_lds[i];
}

template <typename T, int E, int KMAX, bool KTOP1>
static hipError_t launch_split_t(const RouteArgs& a, hipStream_t st) {
  route_valu_split_kernel<T, E, KMAX, KTOP1>
      <<<dim3(a.nb), dim3(kWave * kSplitP), static_cast<size_t>(a.k) * a.E * sizeof(int), st>>>(a);
  return hipGetLastError();
}

template <typename T, int E>
static hipError_t launch_split_e(const RouteArgs& a, hipStream_t st) {
  if (a.kind == 1) return launch_split_t<T, E, 1, true>(a, st);
  if (a.k == 1) return launch_split_t<T, E, 1, false>(a, st);
  if (a.k == 2) return launch_split_t<T, E, 2, false>(a, st);
  if (a.k <= 4) return launch_split_t<T, E, 4, false>(a, st);
  return launch_split_t<T, E, 8, false>(a, st);
}

// the split kernel covers projections with E in {8, 16, 32, 64}, whole 16-byte
// chunks per row and 16-byte aligned x and W
template <typename T>
static bool route_uses_split(const RouteArgs& a) {
  if (a.logits_in || a.d <= 0 || a.d % Chunk<T>::kElems != 0) return false;
  if (a.E != 8 && a.E != 16 && a.E != 32 && a.E != 64) return false;
  return (reinterpret_cast<uintptr_t>(a.x) % 16) == 0 && (reinterpret_cast<uintptr_t>(a.wg) % 16) == 0;
}

template <typename T, int EC, int KMAX, bool KTOP1>
static hipError_t launch_valu_t(const RouteArgs& a, hipStream_t st) {
  route_valu_kernel<T, EC, KMAX, KTOP1><<<dim3(a.nb), dim3(kWave), static_cast<size_t>(a.E) * sizeof(int), st>>>(a);
  return hipGetLastError();
}

template <typename T, int EC>
static hipError_t launch_valu_ec(const RouteArgs& a, hipStream_t st) {
  if (a.kind == 1) return launch_valu_t<T, EC, 1, true>(a, st);
  if (a.k == 1) return launch_valu_t<T, EC, 1, false>(a, st);
  if (a.k == 2) return launch_valu_t<T, EC, 2, false>(a, st);
  if (a.k <= 4) return launch_valu_t<T, EC, 4, false>(a, st);
  return launch_valu_t<T, EC, 8, false>(a, st);
}

template <typename T>
static hipError_t launch_valu_dt(const RouteArgs& a, hipStream_t st) {
  if (route_uses_split<T>(a)) {
    switch (a.E) {
      case 8: return launch_split_e<T, 8>(a, st);
      case 16: return launch_split_e<T, 16>(a, st);
      case 32: return launch_split_e<T, 32>(a, st);
      default: return launch_split_e<T, 64>(a, st);
    }
  }
  if (a.E <= 8) return launch_valu_ec<T, 8>(a, st);
  if (a.E <= 16) return launch_valu_ec<T, 16>(a, st);
  if (a.E <= 32) return launch_valu_ec<T, 32>(a, st);
  return launch_valu_ec<T, 64>(a, st);
}

}  // namespace hetumoe
