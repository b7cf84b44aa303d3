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
  if (a.E <= 8) return launch_valu_ec<T, 8>(a, st);
  if (a.E <= 16) return launch_valu_ec<T, 16>(a, st);
  if (a.E <= 32) return launch_valu_ec<T, 32>(a, st);
  return launch_valu_ec<T, 64>(a, st);
}

}  // namespace hetumoe
