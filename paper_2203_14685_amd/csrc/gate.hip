// Gate kernels for gfx950: step 1 of Algorithm 1 (logit projection, softmax,
// expert selection) and the capacity rule of Sec. 3.1 (each expert keeps at
// most C assignments, handed out rank-major then in token order).
//
// Three launches, all on the caller's stream:
//   route   logits (the projection x.W of Eq. 1, or read from the caller),
//           streaming selection (top-k list, per-group top-1, or hash),
//           softmax weights, and for every 64-token "wave block" a histogram of
//           its (rank, expert) pairs.  Five variants:
//             route_mfma_rs_kernel  bf16, W held in registers (E up to 128,
//                                d 512..2048, d * E up to 128 K):
//                                persistent, projection on
//                                v_mfma_f32_16x16x32_bf16;
//             route_mfma_ph_kernel  bf16, E in {16, 32, 64, 128}, d a multiple
//                                of 512: persistent, W^T staged in LDS per
//                                128 KB K phase;
//             route_mfma_kernel  other bf16 shapes with E a multiple of 16 up
//                                to 128: W staged through LDS per K chunk;
//             route_valu_kernel  any dtype/shape: one thread per token;
//             route_hash_kernel  the hash gate (no projection).
//   scan    one block per expert: exclusive scan of that expert's histogram
//           over (rank, wave block) -> first slot of each run; demand, counts;
//           -1 fill of the unused slot_src entries.
//   assign  one wave per wave block: the rank of each token among the block's
//           tokens with the same expert comes from ballots on the bits of the
//           expert id (ordered, no atomics) -> slots, slot_src.
#include <atomic>

#include "select.hpp"

namespace hetumoe {

// ---------------------------------------------------------------- hash route
// SplitMix64 (Steele, Lea & Flood, OOPSLA 2014): output number n of the
// generator seeded with `seed` is the mixing function applied to seed + n*gamma.
__device__ __forceinline__ uint64_t splitmix64_output(uint64_t seed, uint64_t n) {
  uint64_t z = seed + n * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ __launch_bounds__(kBlock) void route_hash_kernel(RouteArgs a) {
  extern __shared__ int hist_lds[];  // [kWavesPerBlock][E]
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kBlock + tid;
  const bool valid = s < a.S;
  if (valid) {
    const int32_t tid32 = a.token_ids[s];
    int e;
    if (a.hash_table) {
      // table lookup (balanced assignment); ids outside the table or table
      // entries outside [0, E) are out of contract and fold into [0, E)
      const int32_t v = (tid32 >= 0 && tid32 < a.hash_vocab) ? a.hash_table[tid32] : tid32;
      e = ((v % a.E) + a.E) % a.E;
    } else {
      const uint64_t t = static_cast<uint64_t>(static_cast<int64_t>(tid32));
      e = static_cast<int>(splitmix64_output(a.hash_seed, t + 1ull) % static_cast<uint64_t>(a.E));
    }
    a.ids[s] = e;
    a.weights[s] = 1.f;
  }
  const int wb = blockIdx.x * kWavesPerBlock + w;
  wave_block_hist(hist_lds + w * a.E, wb < a.nb, s, valid, wb, a);
}

// ---------------------------------------------------------------- selection on final logits
constexpr int kSelTileE = 128;  // up to this many experts the block's logits are kept in LDS

// One block per 64-token wave block, P lanes per token select on the block's
// final logits.
template <int P, int KMAX, int MODE>  // MODE: 0 top-k, 1 kTop1, 3 hierarchical top-k
__global__ __launch_bounds__(kWave * P) void select_ext_kernel(SelectArgs a) {
  extern __shared__ int hist_lds[];  // [k][E], then (E <= kSelTileE) the block's logits [64][E + 1]
  constexpr int kThreads = kWave * P;
  const int t = threadIdx.x / P, j = threadIdx.x % P;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kWave + t;
  const bool valid = s < a.S;
  const int E = a.E;
  for (int i = threadIdx.x; i < a.k * E; i += kThreads) hist_lds[i] = 0;
  const bool use_tile = E <= kSelTileE;
  float* tile = reinterpret_cast<float*>(hist_lds + a.k * E);
  const bool transform = a.temperature > 0.f || a.fin != a.raw;
  // the block's rows are one contiguous piece of [S, E]: a flat, coalesced pass
  // makes the final logits ((raw + noise) / temperature, or raw), stores them
  // when asked and keeps them in LDS; four loads are issued before their stores
  if (transform || use_tile) {
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kWave * E;
    const int64_t rows = min(static_cast<int64_t>(kWave), a.S - static_cast<int64_t>(blockIdx.x) * kWave);
    const int n = static_cast<int>(rows) * E;
    for (int f0 = threadIdx.x; f0 < n; f0 += 4 * kThreads) {
      float v[4], g[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int f = f0 + u * kThreads;
        v[u] = f < n ? a.raw[base + f] : 0.f;
        g[u] = (f < n && a.noise) ? a.noise[base + f] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int f = f0 + u * kThreads;
        if (f < n) {
          float val = v[u];
          if (a.temperature > 0.f) val = (a.noise ? val + g[u] : val) / a.temperature;
          if (transform) a.fin[base + f] = val;
          if (use_tile) tile[(f / E) * (E + 1) + f % E] = val;
        }
      }
    }
  }
  __syncthreads();
  // invalid tokens select on row 0 (their results are not written)
  const float* lrow = use_tile ? tile + (valid ? t : 0) * (E + 1) : a.fin + (valid ? s : 0) * E;
  if constexpr (MODE == 3) {
    select_token_htopk<P, KMAX>(lrow, E, a.k, E / a.groups, a.normalize, j, valid, a.ids + s * a.k,
                                a.weights + s * a.k, hist_lds);
  } else {
    select_token<P, KMAX, MODE == 1>(lrow, E, a.k, a.normalize, j, valid, a.ids + s * a.k, a.weights + s * a.k,
                                     hist_lds);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < a.k * E; i += kThreads)
    a.hist[static_cast<int64_t>(i) * a.nb + blockIdx.x] = hist_lds[i];
}

template <int P, int KMAX, int MODE>
static hipError_t launch_sel_t(const SelectArgs& a, hipStream_t st) {
  const size_t tile = a.E <= kSelTileE ? static_cast<size_t>(kWave) * (a.E + 1) * sizeof(float) : 0;
  select_ext_kernel<P, KMAX, MODE><<<dim3(static_cast<unsigned>(a.nb)), dim3(kWave * P),
                                     static_cast<size_t>(a.k) * a.E * sizeof(int) + tile, st>>>(a);
  return hipGetLastError();
}

template <int P, int MODE>
static hipError_t launch_sel_m(const SelectArgs& a, hipStream_t st) {
  if (MODE == 1 || a.k == 1) return launch_sel_t<P, 1, MODE>(a, st);
  if (a.k == 2) return launch_sel_t<P, 2, MODE>(a, st);
  if (a.k <= 4) return launch_sel_t<P, 4, MODE>(a, st);
  return launch_sel_t<P, 8, MODE>(a, st);
}

template <int P>
static hipError_t launch_sel_p(const SelectArgs& a, hipStream_t st) {
  if (a.kind == 1) return launch_sel_m<P, 1>(a, st);
  if (a.kind == 3) return launch_sel_m<P, 3>(a, st);
  return launch_sel_m<P, 0>(a, st);
}

hipError_t launch_select_ext(const SelectArgs& a, hipStream_t st) {
  if (a.nb == 0) return hipSuccess;
  // 4 lanes per token when they split the experts evenly (and, for kTop1,
  // agree with the groups), else one
  const bool four = a.E % 4 == 0 && (a.kind != 1 || 4 % a.k == 0 || a.k % 4 == 0);
  return four ? launch_sel_p<4>(a, st) : launch_sel_p<1>(a, st);
}

// ---------------------------------------------------------------- scan kernel
constexpr int kScanThreads = 1024;
constexpr int kScanWaves = kScanThreads / kWave;

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
  for (int i = 0; i < kScanWaves; ++i) {
    const int t = wave_tot[i];
    before += (i < w) ? t : 0;
    total += t;
  }
  __syncthreads();  // wave_tot is reused by the next call
  return v + before;
}

__global__ __launch_bounds__(kScanThreads) void scan_kernel(ScanArgs a) {
  __shared__ int wave_tot[kScanWaves];
  const int e = blockIdx.x;
  int carry = 0;
  if (a.nb <= kScanThreads && a.k <= 8) {
    // every rank's row in one pass: all the loads first, then the scans in
    // rank order
    const int b = threadIdx.x;
    int v[8];
#pragma unroll
    for (int r = 0; r < 8; ++r)
      v[r] = (r < a.k && b < a.nb) ? a.hist[(static_cast<int64_t>(r) * a.E + e) * a.nb + b] : 0;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      if (r >= a.k) break;
      int total;
      const int incl = block_inclusive_scan(v[r], wave_tot, total);
      if (b < a.nb) a.hist[(static_cast<int64_t>(r) * a.E + e) * a.nb + b] = carry + incl - v[r];
      carry += total;
    }
  } else
  for (int r = 0; r < a.k; ++r) {
    int32_t* row = a.hist + (static_cast<int64_t>(r) * a.E + e) * a.nb;
    for (int b0 = 0; b0 < a.nb; b0 += kScanThreads) {
      const int b = b0 + threadIdx.x;
      const int v = (b < a.nb) ? row[b] : 0;
      int total;
      const int incl = block_inclusive_scan(v, wave_tot, total);
      if (b < a.nb) row[b] = carry + incl - v;  // exclusive offset, in place
      carry += total;
    }
  }
  const int kept = min(carry, a.C);
  if (threadIdx.x == 0) {
    a.counts[e] = kept;
    if (a.demand) a.demand[e] = carry;
  }
  for (int c = kept + threadIdx.x; c < a.C; c += kScanThreads) a.slot_src[static_cast<int64_t>(e) * a.C + c] = -1;
}

// ---------------------------------------------------------------- assign kernel
__global__ __launch_bounds__(kBlock) void assign_kernel(AssignArgs a) {
  const int wb = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;  // wave block of this wave
  if (wb >= a.nb) return;
  const int64_t s = static_cast<int64_t>(wb) * kWave + lane_id();
  const bool valid = s < a.S;
  const int k = a.k;
  // ids are in [0, E); invalid lanes use E, so bits of 0..E are compared
  const int nbits = 32 - __clz(a.E);
  const int lane = lane_id();
  for (int r = 0; r < k; ++r) {
    const int e = valid ? a.ids[s * k + r] : a.E;
    // up to 64 experts: lane x loads expert x's offset for this wave block
    // beside the ids, and each lane takes its expert's by a shuffle (no load
    // that waits on the id)
    int off_lane = 0;
    if (a.E <= kWave) off_lane = a.offs[(static_cast<int64_t>(r) * a.E + min(lane, a.E - 1)) * a.nb + wb];
    uint64_t same = ~0ull;
    for (int bit = 0; bit < nbits; ++bit) {
      const bool on = (e >> bit) & 1;
      const uint64_t bal = __ballot(on);
      same &= on ? bal : ~bal;
    }
    const int off_e = a.E <= kWave ? __shfl(off_lane, min(e, a.E - 1), kWave) : 0;
    if (valid) {
      const int base = a.E <= kWave ? off_e : a.offs[(static_cast<int64_t>(r) * a.E + e) * a.nb + wb];
      const int pos = base + popc_below(same);
      const bool kept = pos < a.C;
      a.slots[s * k + r] = kept ? pos : -1;
      if (kept) a.slot_src[static_cast<int64_t>(e) * a.C + pos] = static_cast<int>(s * k + r);
    }
  }
}

// ---------------------------------------------------------------- scan + assign in one launch
// For small histograms (k * E * nb entries): every block takes its own four
// wave blocks and works out their offsets itself, from per-(rank, expert)
// sums over the histogram rows: all earlier ranks of the expert in full, then
// this rank's earlier wave blocks.  The same ranks as the scan kernel followed
// by the assign kernel; block 0 also writes counts and demand, and the blocks
// share marking the empty slots.
constexpr int kFusedMaxEntries = 16384;  // k * E * nb
constexpr int kFusedMaxBlocks = 1024;    // nb
constexpr int kFusedMaxPairs = 1024;     // k * E

__global__ __launch_bounds__(kBlock) void scan_assign_kernel(ScanArgs sa, AssignArgs a) {
  constexpr int kSeg = 16;  // wave blocks per partial sum
  constexpr int kMaxItems = kFusedMaxEntries / kSeg + kFusedMaxPairs;
  __shared__ int tot[kFusedMaxPairs];                    // [k][E] assignments per rank and expert
  __shared__ int pre[kFusedMaxPairs];                    // [k][E] before this block's first wave block
  __shared__ int offs[kWavesPerBlock * kFusedMaxPairs];  // [wave][k][E] offsets of its wave block
  __shared__ int ptot[kMaxItems], ppre[kMaxItems];       // partial sums over kSeg wave blocks
  const int k = a.k, E = a.E, nb = a.nb;
  const int wb0 = blockIdx.x * kWavesPerBlock;
  const int pairs = k * E;
  const int nseg = (nb + kSeg - 1) / kSeg;
  const int items = pairs * nseg;
  for (int it = threadIdx.x; it < items; it += kBlock) {
    const int q = it / nseg, sg = it % nseg;
    const int32_t* row = a.offs + static_cast<int64_t>(q) * nb;  // the histogram (counts)
    int t = 0, p = 0;
#pragma unroll
    for (int j = 0; j < kSeg; ++j) {
      const int b = sg * kSeg + j;
      const int v = b < nb ? row[b] : 0;
      t += v;
      if (b < wb0) p += v;
    }
    ptot[it] = t;
    ppre[it] = p;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < pairs; q += kBlock) {
    int t = 0, p = 0;
    for (int sg = 0; sg < nseg; ++sg) {
      t += ptot[q * nseg + sg];
      p += ppre[q * nseg + sg];
    }
    tot[q] = t;
    pre[q] = p;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < pairs; q += kBlock) {
    const int r = q / E, e = q % E;
    int base = pre[q];
    for (int r2 = 0; r2 < r; ++r2) base += tot[r2 * E + e];  // rank-major: earlier ranks first
    const int32_t* row = a.offs + static_cast<int64_t>(q) * nb;
    for (int w = 0; w < kWavesPerBlock; ++w) {
      offs[w * pairs + q] = base;
      if (wb0 + w < nb) base += row[wb0 + w];
    }
  }
  __syncthreads();
  if (blockIdx.x == 0) {
    for (int e = threadIdx.x; e < E; e += kBlock) {
      int t = 0;
      for (int r = 0; r < k; ++r) t += tot[r * E + e];
      sa.counts[e] = min(t, a.C);
      if (sa.demand) sa.demand[e] = t;
    }
  }
  // empty slots, experts dealt to the blocks in turn
  for (int e = blockIdx.x; e < E; e += gridDim.x) {
    int t = 0;
    for (int r = 0; r < k; ++r) t += tot[r * E + e];
    for (int c = min(t, a.C) + threadIdx.x; c < a.C; c += kBlock) a.slot_src[static_cast<int64_t>(e) * a.C + c] = -1;
  }
  // ranks inside each wave block, as in assign_kernel
  const int w = threadIdx.x / kWave;
  const int wb = wb0 + w;
  if (wb >= nb) return;
  const int64_t s = static_cast<int64_t>(wb) * kWave + lane_id();
  const bool valid = s < a.S;
  const int nbits = 32 - __clz(E);
  for (int r = 0; r < k; ++r) {
    const int e = valid ? a.ids[s * k + r] : E;
    uint64_t same = ~0ull;
    for (int bit = 0; bit < nbits; ++bit) {
      const bool on = (e >> bit) & 1;
      const uint64_t bal = __ballot(on);
      same &= on ? bal : ~bal;
    }
    if (valid) {
      const int pos = offs[w * pairs + r * E + e] + popc_below(same);
      const bool kept = pos < a.C;
      a.slots[s * k + r] = kept ? pos : -1;
      if (kept) a.slot_src[static_cast<int64_t>(e) * a.C + pos] = static_cast<int>(s * k + r);
    }
  }
}

// ---------------------------------------------------------------- launchers
int device_cu_count() {
  // calls may come from several host threads: the cache is atomic (every
  // thread that fills an entry writes the same value)
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

hipError_t launch_route(const RouteArgs& a, hipStream_t st) {
  if (a.nb == 0) return hipSuccess;
  if (a.kind == 2) {
    const unsigned blocks = static_cast<unsigned>((a.nb + kWavesPerBlock - 1) / kWavesPerBlock);
    route_hash_kernel<<<dim3(blocks), dim3(kBlock), static_cast<size_t>(kWavesPerBlock) * a.E * sizeof(int), st>>>(a);
    return hipGetLastError();
  }
#ifndef HETUMOE_ROUTE_VALU_ONLY
  // matrix-core projections (a build with HETUMOE_ROUTE_VALU_ONLY defined, used
  // only to time the vector-ALU routes against them, skips these)
  if (route_uses_mfma_rs(a)) return launch_route_mfma_rs(a, device_cu_count(), st);
  if (route_uses_mfma_ph(a)) return launch_route_mfma_ph(a, device_cu_count(), st);
  if (route_uses_mfma(a)) return launch_route_mfma(a, st);
#endif
  // with logits given, the element type of x and wg is irrelevant
  if (a.dtype == 1 && !a.logits_in) return launch_route_valu_bf16(a, st);
  return launch_route_valu_f32(a, st);
}

hipError_t launch_scan(const ScanArgs& a, hipStream_t st) {
  scan_kernel<<<dim3(a.E), dim3(kScanThreads), 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_scan_assign(const ScanArgs& sa, const AssignArgs& a, hipStream_t st) {
  const int64_t pairs = static_cast<int64_t>(a.k) * a.E;
  if (a.nb > 0 && a.nb <= kFusedMaxBlocks && pairs <= kFusedMaxPairs && pairs * a.nb <= kFusedMaxEntries) {
    const unsigned blocks = static_cast<unsigned>((a.nb + kWavesPerBlock - 1) / kWavesPerBlock);
    scan_assign_kernel<<<dim3(blocks), dim3(kBlock), 0, st>>>(sa, a);
    return hipGetLastError();
  }
  hipError_t err = launch_scan(sa, st);
  if (err != hipSuccess) return err;
  return launch_assign(a, st);
}

hipError_t launch_assign(const AssignArgs& a, hipStream_t st) {
  if (a.nb == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((a.nb + kWavesPerBlock - 1) / kWavesPerBlock);
  assign_kernel<<<dim3(blocks), dim3(kBlock), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace hetumoe
