// Gate kernels for gfx950: step 1 of Algorithm 1 (logit projection, softmax,
// expert selection) and the capacity rule of Sec. 3.1 (each expert keeps at
// most C assignments, handed out rank-major then in token order).
//
// Three launches, all on the caller's stream:
//   route   one thread per token: logits (projection x.W of Eq. 1, or read
//           from the caller), streaming selection (top-k list, per-group
//           top-1, or hash), softmax weights, and a per-block histogram of
//           (rank, expert) pairs.  256 tokens per block.
//   scan    one block per expert: exclusive scan of that expert's histogram
//           entries over (rank, block) order -> the first slot of every
//           (rank, block, expert) run; demand, counts; -1 fill of unused
//           slot_src entries.
//   assign  one thread per token and rank: position inside the block by wave
//           ballots on the bits of the expert id (ordered ranks without
//           atomics) plus a prefix over the block's waves -> slots, slot_src.
#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

// ---------------------------------------------------------------- selection
// Streaming state for one token; experts arrive in increasing index order.
// Order of experts: larger logit first, then lower index.

template <int KMAX>
struct TopkState {
  float tv[KMAX];
  int ti[KMAX];
  float m;     // running max of all logits
  float ssum;  // sum of exp(logit - m) over the logits seen so far
  __device__ void init() {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) { tv[i] = -INFINITY; ti[i] = 0x7fffffff; }
    m = -INFINITY;
    ssum = 0.f;
  }
  __device__ void push(float v, int e) {
    if (v > m) { ssum = ssum * expf(m - v) + 1.f; m = v; }
    else { ssum += expf(v - m); }
    // insertion into the sorted list: the carried pair moves down while it beats
    // the entry it meets
    float cv = v;
    int ci = e;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      // an empty entry (index INT_MAX) always loses, so every reported id is a
      // real expert even for non-finite logits
      bool beats = ti[i] == 0x7fffffff || cv > tv[i] || (cv == tv[i] && ci < ti[i]);
      float ov = tv[i];
      int oi = ti[i];
      tv[i] = beats ? cv : ov;
      ti[i] = beats ? ci : oi;
      cv = beats ? ov : cv;
      ci = beats ? oi : ci;
    }
  }
};

struct Ktop1State {
  int G;       // experts per group
  int g;       // current group
  float bv;    // best (= max) logit of the current group
  int bi;      // its expert index
  float gsum;  // sum of exp(logit - bv) over the group so far
};

// ---------------------------------------------------------------- route kernel
constexpr int kDJ = 64;  // rows of Wg staged in LDS per step

template <typename T, int EC, int KMAX, bool KTOP1>
__global__ __launch_bounds__(kBlock) void route_kernel(RouteArgs a) {
  extern __shared__ int hist_lds[];  // [k][E]
  __shared__ float wg_s[kDJ][EC];

  const int tid = threadIdx.x;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kTokensPerHistBlock + tid;
  const bool valid = s < a.S;
  const int E = a.E, k = a.k;

  for (int i = tid; i < k * E; i += kBlock) hist_lds[i] = 0;
  __syncthreads();

  TopkState<KMAX> tk;
  tk.init();
  Ktop1State kt;
  kt.G = E / k;
  kt.g = 0;
  kt.bv = -INFINITY;
  kt.bi = 0;
  kt.gsum = 0.f;

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
        for (int t = tid; t < kDJ * EC; t += kBlock) {
          const int jj = t / EC, ii = t % EC;
          const int j = j0 + jj, e = e0 + ii;
          wg_s[jj][ii] = (j < a.d && e < E) ? load_elem(wg, static_cast<int64_t>(j) * E + e) : 0.f;
        }
        __syncthreads();
        if (valid) {
          const int jend = min(kDJ, a.d - j0);
          const u32x4* xv = reinterpret_cast<const u32x4*>(xrow + j0);
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
        const int e = e0 + i;
        if (e >= E) break;
        const float v = acc[i];
        if constexpr (KTOP1) {
          const int gstart = kt.g * kt.G;
          if (e == gstart) { kt.bv = v; kt.bi = e; kt.gsum = 1.f; }
          else if (v > kt.bv) { kt.gsum = kt.gsum * expf(kt.bv - v) + 1.f; kt.bv = v; kt.bi = e; }
          else { kt.gsum += expf(v - kt.bv); }
          if (e == gstart + kt.G - 1) {
            a.ids[s * k + kt.g] = kt.bi;
            a.weights[s * k + kt.g] = 1.f / kt.gsum;
            atomicAdd(&hist_lds[kt.g * E + kt.bi], 1);
            ++kt.g;
          }
        } else {
          tk.push(v, e);
        }
      }
    }
  }

  if constexpr (!KTOP1) {
    if (valid) {
      const float top = tk.tv[0];
      float z = 0.f;
      if (a.normalize) {
#pragma unroll
        for (int r = 0; r < KMAX; ++r)
          if (r < k) z += expf(tk.tv[r] - top);
      } else {
        z = tk.ssum * expf(tk.m - top);  // tk.m == top; kept general
      }
      const float inv = 1.f / z;
#pragma unroll
      for (int r = 0; r < KMAX; ++r) {
        if (r < k) {
          a.ids[s * k + r] = tk.ti[r];
          a.weights[s * k + r] = (r == 0 ? 1.f : expf(tk.tv[r] - top)) * inv;
          atomicAdd(&hist_lds[r * E + tk.ti[r]], 1);
        }
      }
    }
  }

  __syncthreads();
  for (int i = tid; i < k * E; i += kBlock) {
    const int r = i / E, e = i % E;
    a.hist[(static_cast<int64_t>(r) * a.nb + blockIdx.x) * E + e] = hist_lds[i];
  }
}

// SplitMix64 (Steele, Lea & Flood, OOPSLA 2014): output number n of the
// generator seeded with `seed` is the mixing function applied to seed + n*gamma.
__device__ __forceinline__ uint64_t splitmix64_output(uint64_t seed, uint64_t n) {
  uint64_t z = seed + n * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ __launch_bounds__(kBlock) void route_hash_kernel(RouteArgs a) {
  extern __shared__ int hist_lds[];  // [E]
  const int tid = threadIdx.x;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kTokensPerHistBlock + tid;
  for (int i = tid; i < a.E; i += kBlock) hist_lds[i] = 0;
  __syncthreads();
  if (s < a.S) {
    const uint64_t t = static_cast<uint64_t>(static_cast<int64_t>(a.token_ids[s]));
    const int e = static_cast<int>(splitmix64_output(a.hash_seed, t + 1ull) % static_cast<uint64_t>(a.E));
    a.ids[s] = e;
    a.weights[s] = 1.f;
    atomicAdd(&hist_lds[e], 1);
  }
  __syncthreads();
  for (int i = tid; i < a.E; i += kBlock) a.hist[static_cast<int64_t>(blockIdx.x) * a.E + i] = hist_lds[i];
}

// ---------------------------------------------------------------- scan kernel
// Block-wide inclusive scan of one int per thread; also returns the total.
__device__ __forceinline__ int block_inclusive_scan(int v, int* wave_tot, int& total) {
  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int u = __shfl_up(v, off, kWave);
    if (lane >= off) v += u;
  }
  if (lane == kWave - 1) wave_tot[w] = v;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) {
    const int t = wave_tot[i];
    before += (i < w) ? t : 0;
    total += t;
  }
  __syncthreads();  // wave_tot may be reused by the next call
  return v + before;
}

__global__ __launch_bounds__(kBlock) void scan_kernel(ScanArgs a) {
  __shared__ int wave_tot[kWavesPerBlock];
  const int e = blockIdx.x;
  const int E = a.E;
  int carry = 0;
  for (int r = 0; r < a.k; ++r) {
    for (int b0 = 0; b0 < a.nb; b0 += kBlock) {
      const int b = b0 + threadIdx.x;
      const int64_t idx = (static_cast<int64_t>(r) * a.nb + b) * E + e;
      const int v = (b < a.nb) ? a.hist[idx] : 0;
      int total;
      const int incl = block_inclusive_scan(v, wave_tot, total);
      if (b < a.nb) a.hist[idx] = carry + incl - v;  // exclusive offset, in place
      carry += total;
    }
  }
  const int kept = min(carry, a.C);
  if (threadIdx.x == 0) {
    a.counts[e] = kept;
    if (a.demand) a.demand[e] = carry;
  }
  for (int c = kept + threadIdx.x; c < a.C; c += kBlock) a.slot_src[static_cast<int64_t>(e) * a.C + c] = -1;
}

// ---------------------------------------------------------------- assign kernel
__global__ __launch_bounds__(kBlock) void assign_kernel(AssignArgs a) {
  extern __shared__ int wave_cnt[];  // [kWavesPerBlock][E]
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int E = a.E, k = a.k;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kTokensPerHistBlock + tid;
  const bool valid = s < a.S;
  // ids are in [0, E); invalid lanes use E, so bits of 0..E are compared
  const int nbits = 32 - __clz(E);
  for (int r = 0; r < k; ++r) {
    for (int i = tid; i < kWavesPerBlock * E; i += kBlock) wave_cnt[i] = 0;
    __syncthreads();
    const int e = valid ? a.ids[s * k + r] : E;
    uint64_t same = ~0ull;
    for (int bit = 0; bit < nbits; ++bit) {
      const bool on = (e >> bit) & 1;
      const uint64_t bal = __ballot(on);
      same &= on ? bal : ~bal;
    }
    const int rank = popc_below(same);
    if (valid && rank == 0) wave_cnt[w * E + e] = __popcll(same);
    __syncthreads();
    if (valid) {
      int pos = a.offs[(static_cast<int64_t>(r) * a.nb + blockIdx.x) * E + e] + rank;
      for (int v = 0; v < w; ++v) pos += wave_cnt[v * E + e];
      const bool kept = pos < a.C;
      a.slots[s * k + r] = kept ? pos : -1;
      if (kept) a.slot_src[static_cast<int64_t>(e) * a.C + pos] = static_cast<int>(s * k + r);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- launchers
template <typename T, int EC, int KMAX, bool KTOP1>
static hipError_t launch_route_t(const RouteArgs& a, hipStream_t st) {
  const size_t shm = static_cast<size_t>(a.k) * a.E * sizeof(int);
  route_kernel<T, EC, KMAX, KTOP1><<<dim3(a.nb), dim3(kBlock), shm, st>>>(a);
  return hipGetLastError();
}

template <typename T, int EC>
static hipError_t launch_route_ec(const RouteArgs& a, hipStream_t st) {
  if (a.kind == 1) return launch_route_t<T, EC, 1, true>(a, st);
  if (a.k == 1) return launch_route_t<T, EC, 1, false>(a, st);
  if (a.k == 2) return launch_route_t<T, EC, 2, false>(a, st);
  if (a.k <= 4) return launch_route_t<T, EC, 4, false>(a, st);
  return launch_route_t<T, EC, 8, false>(a, st);
}

template <typename T>
static hipError_t launch_route_dt(const RouteArgs& a, hipStream_t st) {
  if (a.E <= 8) return launch_route_ec<T, 8>(a, st);
  if (a.E <= 16) return launch_route_ec<T, 16>(a, st);
  if (a.E <= 32) return launch_route_ec<T, 32>(a, st);
  return launch_route_ec<T, 64>(a, st);
}

hipError_t launch_route(const RouteArgs& a, hipStream_t st) {
  if (a.nb == 0) return hipSuccess;
  if (a.kind == 2) {
    route_hash_kernel<<<dim3(a.nb), dim3(kBlock), static_cast<size_t>(a.E) * sizeof(int), st>>>(a);
    return hipGetLastError();
  }
  // with logits given, the element type of x/wg is irrelevant
  if (a.dtype == 1 && !a.logits_in) return launch_route_dt<bf16_t>(a, st);
  return launch_route_dt<float>(a, st);
}

hipError_t launch_scan(const ScanArgs& a, hipStream_t st) {
  scan_kernel<<<dim3(a.E), dim3(kBlock), 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_assign(const AssignArgs& a, hipStream_t st) {
  if (a.nb == 0) return hipSuccess;
  assign_kernel<<<dim3(a.nb), dim3(kBlock), static_cast<size_t>(kWavesPerBlock) * a.E * sizeof(int), st>>>(a);
  return hipGetLastError();
}

}  // namespace hetumoe
