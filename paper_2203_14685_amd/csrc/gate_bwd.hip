// Gradient of the gate (step 1 of Algorithm 1, Eq. 1) for end-to-end training:
// dL from dw through the softmax of Eq. 1 (or its Switch / kTop1 readings) and
// the load-balancing loss, then dW = x^T dL, db = column sums of dL and
// dx = dL W^T.  Sums over tokens run in fixed ranges and a fixed order, so the
// results are bitwise reproducible; there are no atomics on floats.
#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

constexpr int kBwdWaves = 4;
constexpr int kBwdThreads = kBwdWaves * kWave;

template <int P>
__device__ __forceinline__ float group_max(float v) {
#pragma unroll
  for (int m = 1; m < P; m <<= 1) v = fmaxf(v, __shfl_xor(v, m));
  return v;
}

template <int P>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int m = 1; m < P; m <<= 1) v += __shfl_xor(v, m);
  return v;
}

// ---------------------------------------------------------------- first choices
// cnt[e] = number of tokens whose first choice is e (one block; integer atomics
// in LDS, so the counts do not depend on the order).
__global__ __launch_bounds__(1024) void aux_counts_kernel(GateBwdArgs a) {
  extern __shared__ int h[];
  for (int e = threadIdx.x; e < a.E; e += blockDim.x) h[e] = 0;
  __syncthreads();
  for (int64_t s = threadIdx.x; s < a.S; s += blockDim.x) {
    const int e = a.ids[s * a.k];
    if (e >= 0 && e < a.E) atomicAdd(&h[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < a.E; e += blockDim.x) a.cnt[e] = h[e];
}

// ---------------------------------------------------------------- dL
// One wave per 64-token wave block.  P lanes per token (P = E rounded up to a
// power of two, at most 64), EPL experts per lane: lane j of a token holds
// experts j, j + P, ...  Softmax maxima and sums are butterfly reductions over
// the P lanes.
template <int P, int EPL>
__global__ __launch_bounds__(kBwdThreads) void gate_dl_kernel(GateBwdArgs a) {
  constexpr int TP = kWave / P;  // tokens per pass
  const int lane = lane_id();
  const int j = lane % P, sub = lane / P;
  const int64_t wb = static_cast<int64_t>(blockIdx.x) * kBwdWaves + threadIdx.x / kWave;
  if (wb >= a.nb) return;  // no block-wide synchronisation below
  const int E = a.E, k = a.k;
  const bool aux = a.aux_coef != 0.f;
  const bool full_softmax = a.kind == 0 && (a.normalize == 0 || aux);
  const float inv_s = a.S > 0 ? 1.f / static_cast<float>(a.S) : 0.f;
  const float c_aux = a.aux_coef * static_cast<float>(E) * inv_s;
  float f[EPL], psum[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = j + P * i;
    f[i] = (aux && e < E) ? static_cast<float>(a.cnt[e]) * inv_s : 0.f;
    psum[i] = 0.f;
  }

  for (int t0 = 0; t0 < kWave; t0 += TP) {
    const int64_t s = wb * kWave + t0 + sub;
    const bool valid = s < a.S;
    const float* lrow = a.logits + (valid ? s : 0) * E;
    float v[EPL], dl[EPL], p[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = j + P * i;
      v[i] = e < E ? (valid ? lrow[e] : 0.f) : -INFINITY;
      dl[i] = 0.f;
      p[i] = 0.f;
    }
    // chosen experts, their gradients and logits (out-of-range ids are ignored)
    int idr[8];
    float dwr[8], lr[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      idr[r] = -1;
      dwr[r] = 0.f;
      lr[r] = -INFINITY;
      if (r < k && valid) {
        const int e = a.ids[s * k + r];
        if (e >= 0 && e < E) {
          idr[r] = e;
          dwr[r] = a.dw[s * k + r];
          lr[r] = lrow[e];
        }
      }
    }
    float m = 0.f, se = 1.f;
    if (full_softmax) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < EPL; ++i) mx = fmaxf(mx, v[i]);
      m = group_max<P>(mx);
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < EPL; ++i) sum += expf(v[i] - m);
      se = group_sum<P>(sum);
#pragma unroll
      for (int i = 0; i < EPL; ++i) p[i] = expf(v[i] - m) / se;
    }
    if (a.kind == 0 && a.normalize) {
      // softmax over the k chosen logits
      float m2 = -INFINITY;
#pragma unroll
      for (int r = 0; r < 8; ++r) m2 = fmaxf(m2, lr[r]);
      float den = 0.f, w[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        w[r] = idr[r] >= 0 ? expf(lr[r] - m2) : 0.f;
        den += w[r];
      }
      float inner = 0.f;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        w[r] = idr[r] >= 0 ? w[r] / den : 0.f;
        inner += w[r] * dwr[r];
      }
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        if (idr[r] < 0) continue;
        const float g = w[r] * (dwr[r] - inner);
#pragma unroll
        for (int i = 0; i < EPL; ++i)
          if (j + P * i == idr[r]) dl[i] += g;
      }
    } else if (a.kind == 0) {
      // full softmax read at each chosen expert
      float g = 0.f;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        if (idr[r] < 0) continue;
        const float wr = expf(lr[r] - m) / se;
        const float t = dwr[r] * wr;
        g += t;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
          if (j + P * i == idr[r]) dl[i] += t;
      }
#pragma unroll
      for (int i = 0; i < EPL; ++i) dl[i] -= p[i] * g;
    } else {
      // kTop1: softmax within each contiguous group of G experts
      const int G = E / k;
      for (int grp = 0; grp < k; ++grp) {
        const int lo = grp * G, hi = lo + G;
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
          const int e = j + P * i;
          if (e >= lo && e < hi) mx = fmaxf(mx, v[i]);
        }
        const float mg = group_max<P>(mx);
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
          const int e = j + P * i;
          if (e >= lo && e < hi) sum += expf(v[i] - mg);
        }
        const float sg = group_sum<P>(sum);
        // the chosen expert of this group (rank grp)
        int id = -1;
        float dwv = 0.f, lv = 0.f;
#pragma unroll
        for (int r = 0; r < 8; ++r)
          if (r == grp) { id = idr[r]; dwv = dwr[r]; lv = lr[r]; }
        if (id < lo || id >= hi) continue;
        const float scale = dwv * (expf(lv - mg) / sg);
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
          const int e = j + P * i;
          if (e >= lo && e < hi) dl[i] += scale * ((e == id ? 1.f : 0.f) - expf(v[i] - mg) / sg);
        }
      }
    }
    if (aux) {
      float fp = 0.f;
#pragma unroll
      for (int i = 0; i < EPL; ++i) fp += f[i] * p[i];
      fp = group_sum<P>(fp);
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        dl[i] += c_aux * p[i] * (f[i] - fp);
        if (valid) psum[i] += p[i];
      }
    }
    if (valid) {
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const int e = j + P * i;
        if (e < E) a.dl[s * E + e] = dl[i];
      }
    }
  }
  if (aux) {
    // sum over the TP token lanes of the wave, then one partial row per wave block
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      for (int msk = P; msk < kWave; msk <<= 1) psum[i] += __shfl_xor(psum[i], msk);
    if (sub == 0) {
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const int e = j + P * i;
        if (e < E) a.ppart[wb * E + e] = psum[i];
      }
    }
  }
}

// loss = coef * E * sum_e f_e * P_e, P_e summed over wave blocks in order.
__global__ __launch_bounds__(1024) void aux_loss_kernel(GateBwdArgs a) {
  __shared__ float red[1024];
  const int t = threadIdx.x;
  float term = 0.f;
  if (t < a.E && a.S > 0) {
    float pe = 0.f;
    for (int64_t b = 0; b < a.nb; ++b) pe += a.ppart[b * a.E + t];
    const float inv_s = 1.f / static_cast<float>(a.S);
    term = (static_cast<float>(a.cnt[t]) * inv_s) * (pe * inv_s);
  }
  red[t] = term;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  if (t == 0) a.aux_loss[0] = a.aux_coef * static_cast<float>(a.E) * red[0];
}

// ---------------------------------------------------------------- dW, db
// Block (j-tile of 64 columns, token range `split`, expert chunk of EC): x and
// dL tiles of 64 tokens staged in LDS; thread (column jj, expert quarter eg)
// accumulates EC/4 sums.  Partials [split][E][d]; blocks of the first j-tile
// also sum dL for db.
template <typename T, int EC>
__global__ __launch_bounds__(kBwdThreads) void dwg_partial_kernel(GateBwdArgs a) {
  constexpr int EG = EC / 4;
  __shared__ float xs[kWave][kWave + 1];
  __shared__ __align__(16) float ds[kWave][EC];
  const int j0 = blockIdx.x * kWave, split = blockIdx.y, e0 = blockIdx.z * EC;
  const int t = threadIdx.x, jj = t % kWave, eg = t / kWave;
  const T* x = reinterpret_cast<const T*>(a.x);
  const int64_t sb = static_cast<int64_t>(split) * a.split_tokens;
  const int64_t se = min(static_cast<int64_t>(a.S), sb + a.split_tokens);
  float acc[EG];
#pragma unroll
  for (int i = 0; i < EG; ++i) acc[i] = 0.f;
  float bacc = 0.f;
  const bool do_bias = blockIdx.x == 0 && t < EC;
  const bool do_w = a.dwg != nullptr;  // else only db is wanted and x may be absent
  for (int64_t s0 = sb; s0 < se; s0 += kWave) {
    __syncthreads();
    for (int q = t; do_w && q < kWave * kWave; q += kBwdThreads) {
      const int tok = q / kWave, col = q % kWave;
      const int64_t s = s0 + tok;
      const int jx = j0 + col;
      xs[tok][col] = (s < se && jx < a.d) ? load_elem(x, s * a.d + jx) : 0.f;
    }
    for (int q = t; q < kWave * EC; q += kBwdThreads) {
      const int tok = q / EC, ee = q % EC;
      const int64_t s = s0 + tok;
      const int e = e0 + ee;
      ds[tok][ee] = (s < se && e < a.E) ? a.dl[s * a.E + e] : 0.f;
    }
    __syncthreads();
    // a tile's 64 terms are summed on their own, then added to the running sum:
    // the rounding error grows with 64 + (tiles) rather than with the token count
    float tacc[EG];
#pragma unroll
    for (int i = 0; i < EG; ++i) tacc[i] = 0.f;
    for (int tok = 0; do_w && tok < kWave; ++tok) {
      const float xv = xs[tok][jj];
#pragma unroll
      for (int i = 0; i < EG; ++i) tacc[i] = fmaf(xv, ds[tok][eg * EG + i], tacc[i]);
    }
#pragma unroll
    for (int i = 0; i < EG; ++i) acc[i] += tacc[i];
    if (do_bias) {
      float tb = 0.f;
      for (int tok = 0; tok < kWave; ++tok) tb += ds[tok][t];
      bacc += tb;
    }
  }
  const int jw = j0 + jj;
  if (do_w && jw < a.d) {
#pragma unroll
    for (int i = 0; i < EG; ++i) {
      const int e = e0 + eg * EG + i;
      if (e < a.E) a.wpart[(static_cast<int64_t>(split) * a.E + e) * a.d + jw] = acc[i];
    }
  }
  if (do_bias && e0 + t < a.E) a.bpart[static_cast<int64_t>(split) * a.E + e0 + t] = bacc;
}

// dwg[j][e] = sum over splits, in order; dbias likewise.
__global__ __launch_bounds__(kBwdThreads) void dwg_reduce_kernel(GateBwdArgs a) {
  const int64_t n = static_cast<int64_t>(a.E) * a.d;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBwdThreads + threadIdx.x;
  if (a.dwg && idx < n) {
    const int e = static_cast<int>(idx / a.d), jx = static_cast<int>(idx % a.d);
    float v = 0.f;
    for (int sp = 0; sp < a.nsplit; ++sp) v += a.wpart[static_cast<int64_t>(sp) * n + idx];
    a.dwg[static_cast<int64_t>(jx) * a.E + e] = v;
  }
  if (a.dbias && idx < a.E) {
    float v = 0.f;
    for (int sp = 0; sp < a.nsplit; ++sp) v += a.bpart[static_cast<int64_t>(sp) * a.E + idx];
    a.dbias[idx] = v;
  }
}

// ---------------------------------------------------------------- dx
// Block: 64 tokens x 64 columns.  Thread (column jj, token group tg) keeps the
// chunk of W's row j in registers and accumulates 16 tokens; dL tiles are
// staged in LDS and read as broadcasts.
template <typename T, int EC>
__global__ __launch_bounds__(kBwdThreads) void dx_kernel(GateBwdArgs a) {
  constexpr int TPT = kWave / 4;  // tokens per thread
  __shared__ __align__(16) float ds[kWave][EC];
  const int j0 = blockIdx.x * kWave;
  const int64_t s0 = static_cast<int64_t>(blockIdx.y) * kWave;
  const int t = threadIdx.x, jj = t % kWave, tg = t / kWave;
  const int jx = j0 + jj;
  const T* wg = reinterpret_cast<const T*>(a.wg);
  float acc[TPT];
#pragma unroll
  for (int i = 0; i < TPT; ++i) acc[i] = 0.f;
  for (int e0 = 0; e0 < a.E; e0 += EC) {
    __syncthreads();
    for (int q = t; q < kWave * EC; q += kBwdThreads) {
      const int tok = q / EC, ee = q % EC;
      const int64_t s = s0 + tok;
      const int e = e0 + ee;
      ds[tok][ee] = (s < a.S && e < a.E) ? a.dl[s * a.E + e] : 0.f;
    }
    float w[EC];
#pragma unroll
    for (int ee = 0; ee < EC; ++ee)
      w[ee] = (jx < a.d && e0 + ee < a.E) ? load_elem(wg, static_cast<int64_t>(jx) * a.E + e0 + ee) : 0.f;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const float* drow = ds[tg + 4 * i];
#pragma unroll
      for (int ee = 0; ee < EC; ++ee) acc[i] = fmaf(drow[ee], w[ee], acc[i]);
    }
  }
  if (jx >= a.d) return;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    const int64_t s = s0 + tg + 4 * i;
    if (s >= a.S) continue;
    const int64_t o = s * a.d + jx;
    float v = acc[i];
    if (a.dtype == 1) {
      uint16_t* dx = reinterpret_cast<uint16_t*>(a.dx);
      if (a.accumulate) v += __uint_as_float(static_cast<uint32_t>(dx[o]) << 16);
      dx[o] = static_cast<uint16_t>(f32_to_bf16_bits(v));
    } else {
      float* dx = reinterpret_cast<float*>(a.dx);
      if (a.accumulate) v += dx[o];
      dx[o] = v;
    }
  }
}

// ---------------------------------------------------------------- launchers
template <int P, int EPL>
static void launch_dl_t(const GateBwdArgs& a, hipStream_t st) {
  const unsigned blocks = static_cast<unsigned>((a.nb + kBwdWaves - 1) / kBwdWaves);
  gate_dl_kernel<P, EPL><<<dim3(blocks), dim3(kBwdThreads), 0, st>>>(a);
}

hipError_t launch_gate_bwd_dl(const GateBwdArgs& a, hipStream_t st) {
  const bool aux = a.aux_coef != 0.f;
  if (aux) aux_counts_kernel<<<dim3(1), dim3(1024), static_cast<size_t>(a.E) * sizeof(int), st>>>(a);
  if (a.nb > 0) {
    const int E = a.E;
    if (E <= 1) launch_dl_t<1, 1>(a, st);
    else if (E <= 2) launch_dl_t<2, 1>(a, st);
    else if (E <= 4) launch_dl_t<4, 1>(a, st);
    else if (E <= 8) launch_dl_t<8, 1>(a, st);
    else if (E <= 16) launch_dl_t<16, 1>(a, st);
    else if (E <= 32) launch_dl_t<32, 1>(a, st);
    else if (E <= 64) launch_dl_t<64, 1>(a, st);
    else if (E <= 128) launch_dl_t<64, 2>(a, st);
    else if (E <= 256) launch_dl_t<64, 4>(a, st);
    else if (E <= 512) launch_dl_t<64, 8>(a, st);
    else launch_dl_t<64, 16>(a, st);
  }
  if (aux && a.aux_loss) aux_loss_kernel<<<dim3(1), dim3(1024), 0, st>>>(a);
  return hipGetLastError();
}

constexpr int kDwEC = 64;  // experts per dW block
constexpr int kDxEC = 32;  // experts per register chunk in dx

hipError_t launch_gate_bwd_dwg(const GateBwdArgs& a, hipStream_t st) {
  if (a.nsplit > 0) {
    const unsigned jtiles = a.dwg ? static_cast<unsigned>((a.d + kWave - 1) / kWave) : 1u;
    const dim3 grid(jtiles, a.nsplit, (a.E + kDwEC - 1) / kDwEC);
    if (a.dtype == 1) dwg_partial_kernel<bf16_t, kDwEC><<<grid, dim3(kBwdThreads), 0, st>>>(a);
    else dwg_partial_kernel<float, kDwEC><<<grid, dim3(kBwdThreads), 0, st>>>(a);
  }
  const int64_t n = static_cast<int64_t>(a.E) * (a.dwg ? a.d : 1);
  const unsigned blocks = static_cast<unsigned>((n + kBwdThreads - 1) / kBwdThreads);
  if (blocks > 0) dwg_reduce_kernel<<<dim3(blocks), dim3(kBwdThreads), 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_gate_bwd_dx(const GateBwdArgs& a, hipStream_t st) {
  if (a.nb == 0) return hipSuccess;
  const dim3 grid((a.d + kWave - 1) / kWave, a.nb);
  if (a.dtype == 1) dx_kernel<bf16_t, kDxEC><<<grid, dim3(kBwdThreads), 0, st>>>(a);
  else dx_kernel<float, kDxEC><<<grid, dim3(kBwdThreads), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace hetumoe
