// Streaming expert selection and the wave-block histogram shared by the route
// kernels (gate step of Algorithm 1; Eq. 1, Sec. 3.1 kTop1).
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

constexpr int kEmpty = 0x7fffffff;

// ---------------------------------------------------------------- selection
// Streaming state for one token; experts arrive in increasing index order.
// Order of experts: larger logit first, then lower index.

template <int KMAX>
struct TopkState {
  float tv[KMAX];
  int ti[KMAX];
  float m;     // running max of all logits
  float ssum;  // sum of exp(logit - m) over the logits seen so far
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) { tv[i] = -INFINITY; ti[i] = kEmpty; }
    m = -INFINITY;
    ssum = 0.f;
  }
  __device__ __forceinline__ void push(float v, int e) {
    if (v > m) { ssum = ssum * expf(m - v) + 1.f; m = v; }
    else { ssum += expf(v - m); }
    // insertion into the sorted list: the carried pair moves down while it beats
    // the entry it meets; an empty entry always loses, so every reported id is a
    // real expert even for non-finite logits
    float cv = v;
    int ci = e;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      const bool beats = ti[i] == kEmpty || cv > tv[i] || (cv == tv[i] && ci < ti[i]);
      const float ov = tv[i];
      const int oi = ti[i];
      tv[i] = beats ? cv : ov;
      ti[i] = beats ? ci : oi;
      cv = beats ? ov : cv;
      ci = beats ? oi : ci;
    }
  }
  // Writes ids and weights of the first k entries.
  __device__ __forceinline__ void finish(int k, int normalize, int32_t* ids, float* weights) const {
    const float top = tv[0];
    float z = 0.f;
    if (normalize) {
#pragma unroll
      for (int r = 0; r < KMAX; ++r)
        if (r < k) z += expf(tv[r] - top);
    } else {
      z = ssum * expf(m - top);  // m == top for finite logits
    }
    const float inv = 1.f / z;
#pragma unroll
    for (int r = 0; r < KMAX; ++r) {
      if (r < k) {
        ids[r] = ti[r];
        weights[r] = (r == 0 ? 1.f : expf(tv[r] - top)) * inv;
      }
    }
  }
};

// kTop1: k contiguous groups of G experts; the group's best expert and the
// softmax within the group (its weight is 1 / sum exp(l - max)).
struct Ktop1State {
  int G, g, bi;
  float bv, gsum;
  __device__ __forceinline__ void init(int G_) { G = G_; g = 0; bi = 0; bv = -INFINITY; gsum = 0.f; }
  __device__ __forceinline__ void push(float v, int e, int32_t* ids, float* weights) {
    const int gstart = g * G;
    if (e == gstart) { bv = v; bi = e; gsum = 1.f; }
    else if (v > bv) { gsum = gsum * expf(bv - v) + 1.f; bv = v; bi = e; }
    else { gsum += expf(v - bv); }
    if (e == gstart + G - 1) {
      ids[g] = bi;
      weights[g] = 1.f / gsum;
      ++g;
    }
  }
};

// ---------------------------------------------------------------- wave-block histogram
// hist[r][e][wb] = number of tokens of wave block wb whose rank-r choice is e.
// Every wave of the block calls this (it synchronises the block); `active` waves
// own a wave block, `s` is the calling lane's token.  The ids are read back from
// global memory, where the same thread wrote them.
__device__ __forceinline__ void wave_block_hist(int* lds_w, bool active, int64_t s, bool valid, int wb,
                                                const RouteArgs& a) {
  const int lane = lane_id();
  for (int r = 0; r < a.k; ++r) {
    if (active)
      for (int i = lane; i < a.E; i += kWave) lds_w[i] = 0;
    __syncthreads();
    if (active && valid) atomicAdd(&lds_w[a.ids[s * a.k + r]], 1);
    __syncthreads();
    if (active)
      for (int i = lane; i < a.E; i += kWave)
        a.hist[(static_cast<int64_t>(r) * a.E + i) * a.nb + wb] = lds_w[i];
    __syncthreads();
  }
}

}  // namespace hetumoe
