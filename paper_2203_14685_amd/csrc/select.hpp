// Streaming expert selection and the wave-block histogram shared by the route
// kernels (gate step of Algorithm 1; Eq. 1, Sec. 3.1 kTop1).
//
// Order of experts everywhere: larger logit first, then lower expert index.
// Softmax sums are formed online (running maximum, rescaled sum) with the
// hardware exponential (__expf: v_exp_f32 on x*log2(e)); its relative error is
// about |x| * 6e-8 plus one ulp, far inside the 1e-5 weight tolerance.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

constexpr int kEmpty = 0x7fffffff;

// ---------------------------------------------------------------- top-k
template <int KMAX>
struct TopkState {
  float tv[KMAX];
  int ti[KMAX];
  float m;     // running max of the logits seen
  float ssum;  // sum of exp(logit - m) over the logits seen
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) { tv[i] = -INFINITY; ti[i] = kEmpty; }
    m = -INFINITY;
    ssum = 0.f;
  }
  // Sorted insertion: the carried pair moves down while it beats the entry it
  // meets.  An empty entry always loses, so every reported id is a real expert
  // even for non-finite logits.
  __device__ __forceinline__ void insert(float v, int e) {
    float cv = v;
    int ci = e;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      const bool beats = better(cv, ci, tv[i], ti[i]);
      const float ov = tv[i];
      const int oi = ti[i];
      tv[i] = beats ? cv : ov;
      ti[i] = beats ? ci : oi;
      cv = beats ? ov : cv;
      ci = beats ? oi : ci;
    }
  }
  __device__ __forceinline__ void push(float v, int e) {
    if (v > m) { ssum = ssum * __expf(m - v) + 1.f; m = v; }
    else { ssum += __expf(v - m); }
    insert(v, e);
  }
  // (v, i) ranks before (pv, pi): larger logit, then lower index; empty entries last.
  __device__ __forceinline__ static bool better(float v, int i, float pv, int pi) {
    return i != kEmpty && (pi == kEmpty || v > pv || (v == pv && i < pi));
  }
  // Merge with the state of lane (lane ^ mask): afterwards both hold the best
  // KMAX of the union.  The best KMAX of two sorted lists A, B are
  // better-of(A[i], B[KMAX-1-i]), a bitonic sequence; log2(KMAX) half-cleaner
  // stages sort it.
  __device__ __forceinline__ void merge_xor(int mask) {
    float cv[KMAX];
    int ci[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      const float pv = xor_partner(tv[KMAX - 1 - i], mask);
      const int pi = xor_partner(ti[KMAX - 1 - i], mask);
      const bool mine = better(tv[i], ti[i], pv, pi);
      cv[i] = mine ? tv[i] : pv;
      ci[i] = mine ? ti[i] : pi;
    }
#pragma unroll
    for (int st = KMAX / 2; st >= 1; st /= 2) {
#pragma unroll
      for (int i = 0; i < KMAX; ++i) {
        if ((i & st) == 0) {
          const bool keep = better(cv[i], ci[i], cv[i + st], ci[i + st]);
          const float v0 = cv[i], v1 = cv[i + st];
          const int i0 = ci[i], i1 = ci[i + st];
          cv[i] = keep ? v0 : v1;
          ci[i] = keep ? i0 : i1;
          cv[i + st] = keep ? v1 : v0;
          ci[i + st] = keep ? i1 : i0;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < KMAX; ++i) { tv[i] = cv[i]; ti[i] = ci[i]; }
    const float pm = xor_partner(m, mask);
    const float ps = xor_partner(ssum, mask);
    const float nm = fmaxf(m, pm);
    // a side that has seen nothing has m = -inf and ssum = 0: contributes 0
    const float a = (ssum > 0.f) ? ssum * __expf(m - nm) : 0.f;
    const float b = (ps > 0.f) ? ps * __expf(pm - nm) : 0.f;
    ssum = a + b;
    m = nm;
  }
  // Writes ids and weights of the first k entries.
  __device__ __forceinline__ void finish(int k, int normalize, int32_t* ids, float* weights) const {
    const float top = tv[0];
    float z = 0.f;
    if (normalize) {
#pragma unroll
      for (int r = 0; r < KMAX; ++r)
        if (r < k) z += __expf(tv[r] - top);
    } else {
      z = ssum * __expf(m - top);  // m == top for finite logits
    }
    const float inv = 1.f / z;
#pragma unroll
    for (int r = 0; r < KMAX; ++r) {
      if (r < k) {
        ids[r] = ti[r];
        weights[r] = (r == 0 ? 1.f : __expf(tv[r] - top)) * inv;
      }
    }
  }
};

// ---------------------------------------------------------------- kTop1
// Best expert of a run of experts inside one group, with the group softmax sum
// relative to that best logit.
struct GroupBest {
  float bv;    // best (= max) logit
  int bi;      // its expert
  float gsum;  // sum of exp(logit - bv)
  __device__ __forceinline__ void init() { bv = -INFINITY; bi = kEmpty; gsum = 0.f; }
  __device__ __forceinline__ void push(float v, int e) {
    if (bi == kEmpty) { bv = v; bi = e; gsum = 1.f; }
    else if (v > bv) { gsum = gsum * __expf(bv - v) + 1.f; bv = v; bi = e; }
    else { gsum += __expf(v - bv); }
  }
  __device__ __forceinline__ void merge_xor(int mask) {
    const float pv = xor_partner(bv, mask);
    const int pi = xor_partner(bi, mask);
    const float ps = xor_partner(gsum, mask);
    if (pi == kEmpty) return;
    if (bi == kEmpty) { bv = pv; bi = pi; gsum = ps; return; }
    const bool partner_wins = pv > bv || (pv == bv && pi < bi);
    const float nb = partner_wins ? pv : bv;
    gsum = gsum * __expf(bv - nb) + ps * __expf(pv - nb);
    bv = nb;
    bi = partner_wins ? pi : bi;
  }
};

// kTop1 streaming over all experts in index order: k contiguous groups of G;
// each finished group writes its best expert and weight 1 / sum exp(l - max).
struct Ktop1State {
  int G, g;
  GroupBest cur;
  __device__ __forceinline__ void init(int G_) { G = G_; g = 0; cur.init(); }
  __device__ __forceinline__ void push(float v, int e, int32_t* ids, float* weights) {
    cur.push(v, e);
    if (e == (g + 1) * G - 1) {
      ids[g] = cur.bi;
      weights[g] = 1.f / cur.gsum;
      ++g;
      cur.init();
    }
  }
};

// ---------------------------------------------------------------- parallel selection
// Selection for one token by P consecutive lanes of a wave (lane j = 0..P-1 of
// the token streams experts [j*E/P, (j+1)*E/P) of its logit row, then the lanes
// merge by butterfly shuffles).  All P lanes must call this together.  The lane
// that writes an (id, weight) pair also counts it in hist_lds[r][id] (LDS).
template <int P, int KMAX, bool KTOP1>
__device__ __forceinline__ void select_token(const float* lrow, int E, int k, int normalize, int j, bool valid,
                                             int32_t* ids, float* weights, int* hist_lds) {
  const int slice = E / P;
  const int e0 = j * slice;
  if constexpr (!KTOP1) {
    TopkState<KMAX> tk;
    tk.init();
    for (int e = 0; e < slice; ++e) tk.push(lrow[e0 + e], e0 + e);
#pragma unroll
    for (int msk = 1; msk < P; msk <<= 1) tk.merge_xor(msk);
    if (valid && j == 0) {
      tk.finish(k, normalize, ids, weights);
#pragma unroll
      for (int r = 0; r < KMAX; ++r)
        if (r < k) atomicAdd(&hist_lds[r * E + tk.ti[r]], 1);
    }
  } else {
    const int G = E / k;
    if (P % k == 0) {
      // L = P / k lanes per group; lane j's experts lie in group j / L
      const int L = P / k;
      GroupBest gb;
      gb.init();
      for (int e = 0; e < slice; ++e) gb.push(lrow[e0 + e], e0 + e);
      for (int msk = 1; msk < L; msk <<= 1) gb.merge_xor(msk);
      if (valid && j % L == 0) {
        const int grp = j / L;
        ids[grp] = gb.bi;
        weights[grp] = 1.f / gb.gsum;
        atomicAdd(&hist_lds[grp * E + gb.bi], 1);
      }
    } else if (k % P == 0) {
      // each lane's experts are k / P whole groups
      if (valid) {
        for (int grp = e0 / G; grp < (e0 + slice) / G; ++grp) {
          GroupBest gb;
          gb.init();
          for (int e = grp * G; e < (grp + 1) * G; ++e) gb.push(lrow[e], e);
          ids[grp] = gb.bi;
          weights[grp] = 1.f / gb.gsum;
          atomicAdd(&hist_lds[grp * E + gb.bi], 1);
        }
      }
    } else if (valid && j == 0) {
      Ktop1State kt;
      kt.init(G);
      for (int e = 0; e < E; ++e) kt.push(lrow[e], e, ids, weights);
      for (int r = 0; r < k; ++r) atomicAdd(&hist_lds[r * E + ids[r]], 1);
    }
  }
}

// ---------------------------------------------------------------- selection on a compile-time slice
// The same selections for kernels that know E at compile time: lane j's SL =
// E / P logits are read from LDS at once (`lslice` points at them; 8-byte
// aligned for SL = 2, 16-byte aligned from SL = 4 on) and held in registers;
// the maximum comes first and the softmax sum of the slice relative to it
// second, so no step waits on the one before it.
template <int SL>
__device__ __forceinline__ void load_slice(const float* lslice, float (&v)[SL]) {
  if constexpr (SL % 4 == 0) {
#pragma unroll
    for (int i = 0; i < SL; i += 4) {
      const float4 q = *reinterpret_cast<const float4*>(lslice + i);
      v[i] = q.x; v[i + 1] = q.y; v[i + 2] = q.z; v[i + 3] = q.w;
    }
  } else if constexpr (SL == 2) {
    const float2 q = *reinterpret_cast<const float2*>(lslice);
    v[0] = q.x; v[1] = q.y;
  } else {
#pragma unroll
    for (int i = 0; i < SL; ++i) v[i] = lslice[i];
  }
}

template <int SL>
__device__ __forceinline__ float slice_max(const float (&v)[SL]) {
  float mx = v[0];
#pragma unroll
  for (int i = 1; i < SL; ++i) mx = fmaxf(mx, v[i]);
  return mx;
}

template <int SL>
__device__ __forceinline__ float slice_expsum(const float (&v)[SL], float mx) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < SL; ++i) s += __expf(v[i] - mx);
  return s;
}

// Top-k state of a slice: sorted insertion in expert order (an equal logit
// never displaces a lower expert), with the slice's softmax sum.
template <int KMAX, int SL>
__device__ __forceinline__ void topk_of_slice(const float (&v)[SL], int e0, TopkState<KMAX>& tk) {
  tk.init();
  tk.m = slice_max(v);
  tk.ssum = slice_expsum(v, tk.m);
#pragma unroll
  for (int i = 0; i < SL; ++i) tk.insert(v[i], e0 + i);
}

// P lanes per token, each with SL = E / P logits of its row at lrow + j * SL.
template <int P, int KMAX, bool KTOP1, int SL>
__device__ __forceinline__ void select_token_c(const float* lrow, int k, int normalize, int j, bool valid,
                                               int32_t* ids, float* weights, int* hist_lds) {
  constexpr int E = P * SL;
  const int e0 = j * SL;
  if constexpr (!KTOP1) {
    float v[SL];
    load_slice<SL>(lrow + e0, v);
    TopkState<KMAX> tk;
    topk_of_slice<KMAX, SL>(v, e0, tk);
#pragma unroll
    for (int msk = 1; msk < P; msk <<= 1) tk.merge_xor(msk);
    if (valid && j == 0) {
      tk.finish(k, normalize, ids, weights);
#pragma unroll
      for (int r = 0; r < KMAX; ++r)
        if (r < k) atomicAdd(&hist_lds[r * E + tk.ti[r]], 1);
    }
  } else if (P % k == 0) {
    // L = P / k lanes per group; lane j's experts lie in group j / L
    const int L = P / k;
    float v[SL];
    load_slice<SL>(lrow + e0, v);
    GroupBest gb;
    gb.bv = v[0];
    gb.bi = e0;
#pragma unroll
    for (int i = 1; i < SL; ++i) {
      const bool up = v[i] > gb.bv;  // strict: the lower expert keeps a tie
      gb.bv = up ? v[i] : gb.bv;
      gb.bi = up ? e0 + i : gb.bi;
    }
    gb.gsum = slice_expsum(v, gb.bv);
    for (int msk = 1; msk < L; msk <<= 1) gb.merge_xor(msk);
    if (valid && j % L == 0) {
      const int grp = j / L;
      ids[grp] = gb.bi;
      weights[grp] = 1.f / gb.gsum;
      atomicAdd(&hist_lds[grp * E + gb.bi], 1);
    }
  } else {
    select_token<P, KMAX, true>(lrow, E, k, normalize, j, valid, ids, weights, hist_lds);
  }
}

// ---------------------------------------------------------------- wave-block histogram
// hist[r][e][wb] = number of tokens of wave block wb whose rank-r choice is e.
// Every wave of the block calls this (it synchronises the block); `active` waves
// own a wave block, `s` is the calling lane's token.  The ids are read back from
// global memory, where the same thread wrote them.
// Hierarchical top-k for one token by P consecutive lanes (Sec. 3.1, H Topk):
// the best expert over all E (with the full softmax sum), its group of Gs
// contiguous experts, then the k best experts of that group.  Weights: softmax
// over the k chosen (normalize) or the full softmax at each of them.
template <int P, int KMAX>
__device__ __forceinline__ void select_token_htopk(const float* lrow, int E, int k, int Gs, int normalize, int j,
                                                   bool valid, int32_t* ids, float* weights, int* hist_lds) {
  const int slice = E / P;
  const int e0 = j * slice;
  TopkState<1> t1;
  t1.init();
  for (int e = 0; e < slice; ++e) t1.push(lrow[e0 + e], e0 + e);
#pragma unroll
  for (int msk = 1; msk < P; msk <<= 1) t1.merge_xor(msk);
  const int best = t1.ti[0] == kEmpty ? 0 : t1.ti[0];
  const int lo = (best / Gs) * Gs, hi = lo + Gs;
  TopkState<KMAX> tk;
  tk.init();
  for (int e = 0; e < slice; ++e) {
    const int ee = e0 + e;
    if (ee >= lo && ee < hi) tk.insert(lrow[ee], ee);
  }
#pragma unroll
  for (int msk = 1; msk < P; msk <<= 1) tk.merge_xor(msk);
  // the group holds the overall best: the full softmax sum relative to it
  tk.m = t1.m;
  tk.ssum = t1.ssum;
  if (valid && j == 0) {
    tk.finish(k, normalize, ids, weights);
#pragma unroll
    for (int r = 0; r < KMAX; ++r)
      if (r < k) atomicAdd(&hist_lds[r * E + tk.ti[r]], 1);
  }
}

// Hierarchical top-k on a compile-time slice (see select_token_c).
template <int P, int KMAX, int SL>
__device__ __forceinline__ void select_token_htopk_c(const float* lrow, int k, int Gs, int normalize, int j,
                                                     bool valid, int32_t* ids, float* weights, int* hist_lds) {
  constexpr int E = P * SL;
  const int e0 = j * SL;
  float v[SL];
  load_slice<SL>(lrow + e0, v);
  TopkState<1> t1;
  topk_of_slice<1, SL>(v, e0, t1);
#pragma unroll
  for (int msk = 1; msk < P; msk <<= 1) t1.merge_xor(msk);
  const int best = t1.ti[0] == kEmpty ? 0 : t1.ti[0];
  const int lo = (best / Gs) * Gs, hi = lo + Gs;
  TopkState<KMAX> tk;
  tk.init();
  // experts outside the group go in as empty entries, which never displace
  // anything (no branch per logit)
#pragma unroll
  for (int i = 0; i < SL; ++i) {
    const int ee = e0 + i;
    const bool in = ee >= lo && ee < hi;
    tk.insert(in ? v[i] : -INFINITY, in ? ee : kEmpty);
  }
#pragma unroll
  for (int msk = 1; msk < P; msk <<= 1) tk.merge_xor(msk);
  // the group holds the overall best: the full softmax sum relative to it
  tk.m = t1.m;
  tk.ssum = t1.ssum;
  if (valid && j == 0) {
    tk.finish(k, normalize, ids, weights);
#pragma unroll
    for (int r = 0; r < KMAX; ++r)
      if (r < k) atomicAdd(&hist_lds[r * E + tk.ti[r]], 1);
  }
}

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
