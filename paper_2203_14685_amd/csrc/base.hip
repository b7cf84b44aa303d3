// BASE layer gate (Sec. 3.1, BASE Layer): the balanced assignment that gives
// every expert exactly c = S / E tokens and maximises the summed score
// L[s, a_s], solved by an auction (Bertsekas) on the gate logits.
//
// Each expert is one object of capacity c with a price p_e.  In a round every
// unassigned token s bids for its best expert e1 = argmax_e (L[s,e] - p_e) the
// amount L[s,e1] - v2 + eps, v2 the best L[s,e] - p_e over the other experts.
// Each expert keeps the c best of its holders and its new bidders, in the total
// order (bid descending, token ascending), evicts the rest and, once full, sets
// its price to its c-th best bid.  A held token's bid is at least its expert's
// price and prices only rise, so every held token stays within eps of its best
// net value (eps-complementary slackness); when no token is unassigned the
// assignment is within S * eps of the optimum (the dual bound).  eps is lowered
// in phases (eps-scaling: prices kept, holders cleared).  Prices and bids are
// fp64.  Every step runs in a fixed order, so results are bitwise reproducible.
#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

constexpr int kBaseThreads = 1024;  // resolve: one block per expert

// (v, t) before (w, u): larger bid, then lower token
__device__ __forceinline__ bool base_before(double v, int t, double w, int u) {
  return v > w || (v == w && t < u);
}

// ---------------------------------------------------------------- score range
__global__ __launch_bounds__(kBaseThreads) void base_minmax_kernel(BaseArgs a) {
  __shared__ float mx[kBaseThreads], mn[kBaseThreads];
  float hi = -INFINITY, lo = INFINITY;
  int nan = 0;
  const int64_t n = static_cast<int64_t>(a.S) * a.E;
  for (int64_t i = threadIdx.x; i < n; i += kBaseThreads) {
    const float v = a.logits[i];
    hi = fmaxf(hi, v);
    lo = fminf(lo, v);
    nan |= v != v;
  }
  mx[threadIdx.x] = hi;
  mn[threadIdx.x] = lo;
  nan = __syncthreads_or(nan);
  for (int w = kBaseThreads / 2; w > 0; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w) {
      mx[threadIdx.x] = fmaxf(mx[threadIdx.x], mx[threadIdx.x + w]);
      mn[threadIdx.x] = fminf(mn[threadIdx.x], mn[threadIdx.x + w]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    a.range[0] = nan ? NAN : mn[0];
    a.range[1] = mx[0];
  }
}

// ---------------------------------------------------------------- phase start
// every token unassigned, holders cleared; prices start at 0 in the first phase
__global__ __launch_bounds__(kBlock) void base_reset_kernel(BaseArgs a, int first) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i < a.S) a.assign[i] = -1;
  if (i < a.E) {
    a.hold_n[i] = 0;
    if (first) a.price[i] = 0.0;
  }
}

__global__ __launch_bounds__(kWave) void base_zero_counts_kernel(int32_t* cnt, int n) {
  if (static_cast<int>(threadIdx.x) < n) cnt[threadIdx.x] = 0;
}

// ---------------------------------------------------------------- bids
// One thread per token; cnt counts the tokens unassigned at the round's start.
__global__ __launch_bounds__(kBlock) void base_bid_kernel(BaseArgs a, double eps, int32_t* cnt) {
  extern __shared__ double price[];  // [E]
  __shared__ int nblk;
  for (int e = threadIdx.x; e < a.E; e += kBlock) price[e] = a.price[e];
  if (threadIdx.x == 0) nblk = 0;
  __syncthreads();
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (s < a.S) {
    if (a.assign[s] < 0) {
      const float* row = a.logits + s * a.E;
      double v1 = -INFINITY, v2 = -INFINITY;
      int e1 = 0;
      for (int e = 0; e < a.E; ++e) {
        const double v = static_cast<double>(row[e]) - price[e];
        if (v > v1) {
          v2 = v1;
          v1 = v;
          e1 = e;
        } else if (v > v2) {
          v2 = v;
        }
      }
      if (a.E == 1) v2 = v1;  // one expert: bid just above its price
      a.bid_e[s] = e1;
      a.bid_v[s] = static_cast<double>(row[e1]) - v2 + eps;
      atomicAdd(&nblk, 1);
    } else {
      a.bid_e[s] = -1;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0 && nblk > 0) atomicAdd(cnt, nblk);
}

// ---------------------------------------------------------------- resolve
// n a power of two, at most 2 * kBaseThreads: sorted into (bid desc, token asc)
__device__ __forceinline__ void base_sort(double* v, int* t, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size / 2; stride > 0; stride >>= 1) {
      const int i = threadIdx.x;
      if (i < n / 2) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = (lo & size) == 0 || size == n;
        const bool swap = desc ? base_before(v[hi], t[hi], v[lo], t[lo]) : base_before(v[lo], t[lo], v[hi], t[hi]);
        if (swap) {
          const double tv = v[lo];
          v[lo] = v[hi];
          v[hi] = tv;
          const int tt = t[lo];
          t[lo] = t[hi];
          t[hi] = tt;
        }
      }
      __syncthreads();
    }
  }
}

// One block per expert.  Bidders are collected in token order, at most
// kBaseCand per round (later ones stay unassigned and bid again), sorted, and
// merged with the sorted holders by rank; ranks below c survive.
__global__ __launch_bounds__(kBaseThreads) void base_resolve_kernel(BaseArgs a) {
  extern __shared__ double base_lds[];
  const int c = a.cap;
  double* hv = base_lds;                            // holders [c]
  double* bv = hv + c;                              // bidders [kBaseCand]
  int* ht = reinterpret_cast<int*>(bv + kBaseCand); // [c]
  int* bt = ht + c;                                 // [kBaseCand]
  __shared__ int wave_cnt[kBaseThreads / kWave];
  __shared__ int nb_total;
  const int e = blockIdx.x;
  const int64_t base = static_cast<int64_t>(e) * c;
  const int nh = a.hold_n[e];
  for (int i = threadIdx.x; i < nh; i += kBaseThreads) {
    hv[i] = a.hold_v[base + i];
    ht[i] = a.hold_t[base + i];
  }
  if (threadIdx.x == 0) nb_total = 0;
  __syncthreads();
  const int lane = lane_id(), w = threadIdx.x / kWave;
  for (int64_t s0 = 0; s0 < a.S; s0 += kBaseThreads) {
    const int have = nb_total;  // uniform: written before the last barrier
    if (have >= kBaseCand) break;
    const int64_t s = s0 + threadIdx.x;
    const bool mine = s < a.S && a.bid_e[s] == e;
    const uint64_t ballot = __ballot(mine);
    if (lane == 0) wave_cnt[w] = __popcll(ballot);
    __syncthreads();
    int before = 0;
    for (int i = 0; i < w; ++i) before += wave_cnt[i];
    const int pos = have + before + popc_below(ballot);
    if (mine && pos < kBaseCand) {
      bv[pos] = a.bid_v[s];
      bt[pos] = static_cast<int>(s);
    }
    int tot = 0;
    for (int i = 0; i < kBaseThreads / kWave; ++i) tot += wave_cnt[i];
    __syncthreads();
    if (threadIdx.x == 0) nb_total = min(kBaseCand, have + tot);
    __syncthreads();
  }
  const int nb = nb_total;
  if (nb == 0) return;  // uniform: nothing changes for this expert
  int np2 = 1;
  while (np2 < nb) np2 <<= 1;
  for (int i = nb + threadIdx.x; i < np2; i += kBaseThreads) {
    bv[i] = -INFINITY;
    bt[i] = 0x7fffffff;
  }
  __syncthreads();
  base_sort(bv, bt, np2);
  // rank of each entry in the union of the two sorted, disjoint lists
  for (int i = threadIdx.x; i < nh; i += kBaseThreads) {
    int lo = 0, hi = nb;  // bidders ahead of holder i
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (base_before(bv[mid], bt[mid], hv[i], ht[i])) lo = mid + 1;
      else hi = mid;
    }
    const int r = i + lo;
    if (r < c) {
      a.hold_v[base + r] = hv[i];
      a.hold_t[base + r] = ht[i];
      if (r == c - 1) a.price[e] = hv[i];
    } else {
      a.assign[ht[i]] = -1;  // evicted
    }
  }
  for (int j = threadIdx.x; j < nb; j += kBaseThreads) {
    int lo = 0, hi = nh;  // holders ahead of bidder j
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (base_before(hv[mid], ht[mid], bv[j], bt[j])) lo = mid + 1;
      else hi = mid;
    }
    const int r = j + lo;
    if (r < c) {
      a.hold_v[base + r] = bv[j];
      a.hold_t[base + r] = bt[j];
      a.assign[bt[j]] = e;
      if (r == c - 1) a.price[e] = bv[j];
    }
  }
  if (threadIdx.x == 0) a.hold_n[e] = min(c, nh + nb);
}

// ---------------------------------------------------------------- outputs
// ids, weights (sigmoid of the score) and the wave-block histogram [E, nb]
// that the scan and assign kernels turn into slots
__global__ __launch_bounds__(kBlock) void base_finish_kernel(BaseArgs a) {
  extern __shared__ int hist_lds[];  // [kWavesPerBlock, E]
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = lane_id();
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kBlock + tid;
  const bool valid = s < a.S;
  int e = 0;
  if (valid) {
    e = a.assign[s];
    a.ids[s] = e;
    a.weights[s] = 1.f / (1.f + expf(-a.logits[s * a.E + e]));
  }
  const int wb = blockIdx.x * kWavesPerBlock + w;
  int* lds = hist_lds + w * a.E;
  for (int i = lane; i < a.E; i += kWave) lds[i] = 0;
  __syncthreads();
  if (valid) atomicAdd(&lds[e], 1);
  __syncthreads();
  if (wb < a.nb)
    for (int i = lane; i < a.E; i += kWave) a.hist[static_cast<int64_t>(i) * a.nb + wb] = lds[i];
}

// ---------------------------------------------------------------- driver
size_t base_resolve_lds(int cap) { return static_cast<size_t>(cap + kBaseCand) * (sizeof(double) + sizeof(int)); }

hipError_t run_base_auction(const BaseArgs& a, hipStream_t st, BaseStats* stats) {
  hipError_t err;
  *stats = BaseStats{};
  if (a.S == 0) return hipSuccess;
  const unsigned tok_blocks = static_cast<unsigned>((a.S + kBlock - 1) / kBlock);
  base_minmax_kernel<<<1, kBaseThreads, 0, st>>>(a);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  float range[2] = {0.f, 0.f};
  if ((err = hipMemcpyAsync(range, a.range, sizeof(range), hipMemcpyDeviceToHost, st)) != hipSuccess) return err;
  if ((err = hipStreamSynchronize(st)) != hipSuccess) return err;
  const double spread = static_cast<double>(range[1]) - static_cast<double>(range[0]);
  if (!(spread < INFINITY)) {  // inf or nan among the scores
    stats->bad_scores = 1;
    return hipSuccess;
  }
  // eps: a quarter of the score range, divided by kBaseEpsStep per phase down
  // to the range times kBaseEpsEnd (one phase when every score is equal: every
  // balanced assignment is then optimal)
  const double eps_end = spread > 0.0 ? spread * kBaseEpsEnd : 1.0;
  double eps = spread > 0.0 ? spread / 4.0 : eps_end;
  constexpr int kBatch = 8;  // rounds between reads of the unassigned counts
  for (;;) {
    base_reset_kernel<<<tok_blocks, kBlock, 0, st>>>(a, stats->phases == 0);
    int rounds = 0;
    bool done = false;
    while (!done) {
      base_zero_counts_kernel<<<1, kWave, 0, st>>>(a.counts, kBatch);
      for (int r = 0; r < kBatch; ++r) {
        base_bid_kernel<<<tok_blocks, kBlock, static_cast<size_t>(a.E) * sizeof(double), st>>>(a, eps, a.counts + r);
        base_resolve_kernel<<<static_cast<unsigned>(a.E), kBaseThreads, base_resolve_lds(a.cap), st>>>(a);
      }
      if ((err = hipGetLastError()) != hipSuccess) return err;
      int32_t cnt[kBatch];
      if ((err = hipMemcpyAsync(cnt, a.counts, sizeof(cnt), hipMemcpyDeviceToHost, st)) != hipSuccess) return err;
      if ((err = hipStreamSynchronize(st)) != hipSuccess) return err;
      // a round that began with no unassigned token ends the phase
      for (int r = 0; r < kBatch && !done; ++r) {
        if (cnt[r] == 0) done = true;
        else ++rounds;
      }
      if (!done && rounds >= a.max_rounds) {
        stats->rounds += rounds;
        stats->not_converged = 1;
        return hipSuccess;
      }
    }
    stats->rounds += rounds;
    stats->phases += 1;
    stats->eps = eps;
    if (eps <= eps_end) break;
    eps = fmax(eps / kBaseEpsStep, eps_end);
  }
  base_finish_kernel<<<tok_blocks, kBlock, static_cast<size_t>(kWavesPerBlock) * a.E * sizeof(int), st>>>(a);
  return hipGetLastError();
}

}  // namespace hetumoe
