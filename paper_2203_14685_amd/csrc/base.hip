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
//
// The auction's control lives on the device: round r reads the state block
// state[r & 1] and the resolve kernel's block 0 writes state[(r + 1) & 1], so
// the host only enqueues rounds (paced by a progress word the device writes to
// pinned host memory, or a fixed number of them in the asynchronous form).
// Rounds enqueued after the auction has finished return at once.
#include <chrono>
#include <cstdlib>

#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

constexpr int kBaseThreads = 1024;                  // resolve: one block per expert
constexpr int kBaseSortFrom = 256;                  // more bidders than this: sort instead of counting
constexpr int kBaseWaves = kBaseThreads / kWave;    // 16
constexpr int kBaseIters = 32;                      // token tiles of kBaseThreads per collection pass

// (v, t) before (w, u): larger bid, then lower token
__device__ __forceinline__ bool base_before(double v, int t, double w, int u) {
  return v > w || (v == w && t < u);
}

// ---------------------------------------------------------------- set-up
// Score range, in two steps: per-block minimum, maximum and a NaN / infinity
// flag over a grid-strided share of the scores, then one block that reduces
// them, derives the eps schedule and writes the first state.  A NaN or
// infinite score ends the auction before it starts (failed = 2).
__global__ __launch_bounds__(kBaseThreads) void base_range_kernel(BaseArgs a) {
  __shared__ float mx[kBaseThreads], mn[kBaseThreads];
  float hi = -INFINITY, lo = INFINITY;
  int bad = 0;
  const int64_t n = static_cast<int64_t>(a.S) * a.E;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBaseThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(kBaseRangeBlocks) * kBaseThreads) {
    const float v = a.logits[i];
    hi = fmaxf(hi, v);
    lo = fminf(lo, v);
    bad |= !(fabsf(v) <= __FLT_MAX__);  // NaN or infinite
  }
  mx[threadIdx.x] = hi;
  mn[threadIdx.x] = lo;
  bad = __syncthreads_or(bad);
  for (int w = kBaseThreads / 2; w > 0; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w) {
      mx[threadIdx.x] = fmaxf(mx[threadIdx.x], mx[threadIdx.x + w]);
      mn[threadIdx.x] = fminf(mn[threadIdx.x], mn[threadIdx.x + w]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    a.range_part[blockIdx.x] = mn[0];
    a.range_part[kBaseRangeBlocks + blockIdx.x] = mx[0];
    a.range_part[2 * kBaseRangeBlocks + blockIdx.x] = bad ? 1.f : 0.f;
  }
}

__global__ __launch_bounds__(kBaseRangeBlocks) void base_init_kernel(BaseArgs a) {
  __shared__ float mx[kBaseRangeBlocks], mn[kBaseRangeBlocks];
  const int t = threadIdx.x;
  mn[t] = a.range_part[t];
  mx[t] = a.range_part[kBaseRangeBlocks + t];
  const int bad = __syncthreads_or(a.range_part[2 * kBaseRangeBlocks + t] != 0.f);
  for (int w = kBaseRangeBlocks / 2; w > 0; w >>= 1) {
    if (t < w) {
      mx[t] = fmaxf(mx[t], mx[t + w]);
      mn[t] = fminf(mn[t], mn[t + w]);
    }
    __syncthreads();
  }
  if (t == 0) {
    const double spread = static_cast<double>(mx[0]) - static_cast<double>(mn[0]);
    BaseState st{};
    // eps: a quarter of the score range, divided by kBaseEpsStep per phase down
    // to the range times kBaseEpsEnd (one phase when every score is equal:
    // every balanced assignment is then optimal)
    st.eps_end = spread > 0.0 ? spread * kBaseEpsEnd : 1.0;
    st.eps = spread > 0.0 ? spread / 4.0 : st.eps_end;
    st.failed = bad ? 2 : 0;
    st.done = bad ? 1 : 0;
    a.state[0] = st;
    a.state[1] = st;
    for (int i = 0; i < 4; ++i) a.counts[i] = 0;
  }
}

// every token unassigned, holders cleared, prices 0, no bids counted
__global__ __launch_bounds__(kBlock) void base_reset_kernel(BaseArgs a) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i < a.S) a.assign[i] = -1;
  if (i < a.E) {
    a.hold_n[i] = 0;
    a.bid_cnt[i] = 0;
    a.price[i] = 0.0;
  }
}

// The bid of token t with G lanes over experts (an aligned group of G lanes
// per token, G <= 16 so that the butterflies stay in a row of the wave): the
// best value (lower expert on ties) and the best other value by butterflies
// over (value, expert); max is exact, so this equals the sequential scan of
// base_bid_kernel.  Every lane of the group returns the same expert and bid.
template <int G>
__device__ __forceinline__ void base_group_bid(const BaseArgs& a, const double* pr, double eps, int t, int sub,
                                               int& e_out, double& bid_out) {
  static_assert(G >= 1 && G <= 16 && (G & (G - 1)) == 0, "G a power of two up to 16");
  const float* row = a.logits + static_cast<int64_t>(t) * a.E;
  double v1 = -INFINITY, v2 = -INFINITY, l1 = 0.0;
  int e1 = 0x7fffffff;
  for (int e0 = 0; e0 < a.E; e0 += 8 * G) {
    float lv[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {  // loads issued together (clamped: past E reads expert 0, skipped)
      const int e = e0 + q * G + sub;
      lv[q] = row[e < a.E ? e : 0];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int e = e0 + q * G + sub;
      if (e >= a.E) continue;
      const double v = static_cast<double>(lv[q]) - pr[e];
      if (v > v1) {
        v2 = v1;
        v1 = v;
        e1 = e;
        l1 = static_cast<double>(lv[q]);
      } else if (v > v2) {
        v2 = v;
      }
    }
  }
#pragma unroll
  for (int off = 1; off < G; off <<= 1) {
    const double ov1 = xor_partner(v1, off), ov2 = xor_partner(v2, off);
    const double ol1 = xor_partner(l1, off);
    const int oe1 = xor_partner(e1, off);
    if (ov1 > v1 || (ov1 == v1 && oe1 < e1)) {
      v2 = fmax(ov2, v1);
      v1 = ov1;
      e1 = oe1;
      l1 = ol1;
    } else {
      v2 = fmax(v2, ov1);
    }
  }
  if (a.E == 1) v2 = v1;
  e_out = e1;
  bid_out = l1 - v2 + eps;
}

// ---------------------------------------------------------------- bids
// One thread per token.  counts[r & 1] receives the number of tokens unassigned
// at the round's start, bid_cnt[e] the bidders of expert e.
template <bool VEC>
__global__ __launch_bounds__(kBlock) void base_bid_kernel(BaseArgs a, int r) {
  // the token's assignment and the first kBlock prices are read with the
  // state: a launch waits for one memory round trip before its first decision
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const int asg = a.assign[s < a.S ? s : 0];
  const double p0 = a.price[threadIdx.x < a.E ? threadIdx.x : 0];
  const BaseState st = a.state[r & 1];
  if (st.done) return;
  extern __shared__ double price[];  // [E], then int ecnt[E]
  int* ecnt = reinterpret_cast<int*>(price + a.E);
  __shared__ int nblk;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    a.counts[(r + 1) & 1] = 0;  // for the next round
    a.counts[2 + (r & 1)] = 0;  // slots this round's resolve step fills
  }
  for (int e = threadIdx.x; e < a.E; e += kBlock) {
    price[e] = e < kBlock ? p0 : a.price[e];
    ecnt[e] = 0;
  }
  __shared__ int lst[16], nlst, boff;
  if (threadIdx.x == 0) {
    nblk = 0;
    nlst = 0;
  }
  int myrank = -1;  // this thread's bidder's place in the block's share of the round's list
  int mytok = 0;
  const bool bidder = s < a.S && asg < 0;
  if (s < a.S && !bidder) a.bid_e[s] = -1;
  const int nbb = __syncthreads_count(bidder);
  if (nbb == 0) return;  // no bidder in this block
  if (nbb <= 16) {
    // few bidders (the later rounds of a phase): 16 lanes over the experts each
    if (bidder) lst[atomicAdd(&nlst, 1)] = threadIdx.x;
    __syncthreads();
    const int g = threadIdx.x / 16;
    if (g < nbb) {  // uniform in each group of 16 lanes
      const int64_t t = static_cast<int64_t>(blockIdx.x) * kBlock + lst[g];
      int e1;
      double bid;
      base_group_bid<16>(a, price, st.eps, static_cast<int>(t), threadIdx.x % 16, e1, bid);
      if (threadIdx.x % 16 == 0) {
        a.bid_e[t] = e1;
        a.bid_v[t] = bid;
        atomicAdd(&ecnt[e1], 1);
        myrank = atomicAdd(&nblk, 1);
        mytok = static_cast<int>(t);
      }
    }
  } else if (bidder) {
    const float* row = a.logits + s * a.E;
    double v1 = -INFINITY, v2 = -INFINITY;
    int e1 = 0;
    auto take = [&](float l, int e) {
      const double v = static_cast<double>(l) - price[e];
      if (v > v1) {
        v2 = v1;
        v1 = v;
        e1 = e;
      } else if (v > v2) {
        v2 = v;
      }
    };
    if constexpr (VEC) {
      const float4* r4 = reinterpret_cast<const float4*>(row);
      const int nq = a.E / 4;
      for (int q0 = 0; q0 < nq; q0 += 16) {  // 64 experts' loads issued together
        float4 l[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) l[q] = r4[q0 + q < nq ? q0 + q : 0];
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          if (q0 + q >= nq) break;
          take(l[q].x, 4 * (q0 + q));
          take(l[q].y, 4 * (q0 + q) + 1);
          take(l[q].z, 4 * (q0 + q) + 2);
          take(l[q].w, 4 * (q0 + q) + 3);
        }
      }
    } else {
      for (int e = 0; e < a.E; ++e) take(row[e], e);
    }
    if (a.E == 1) v2 = v1;  // one expert: bid just above its price
    a.bid_e[s] = e1;
    a.bid_v[s] = static_cast<double>(row[e1]) - v2 + st.eps;
    atomicAdd(&ecnt[e1], 1);
    myrank = atomicAdd(&nblk, 1);
    mytok = static_cast<int>(s);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < a.E; e += kBlock)
    if (ecnt[e] > 0) atomicAdd(&a.bid_cnt[e], ecnt[e]);
  // the block's places in the round's bidder list
  if (threadIdx.x == 0) boff = atomicAdd(&a.counts[r & 1], nblk);
  __syncthreads();
  if (myrank >= 0) a.blist[boff + myrank] = mytok;
}

// ---------------------------------------------------------------- resolve
// n a power of two, at most 2 * kBaseThreads: (v, t) pairs sorted into
// (bid desc, token asc) by a bitonic network, a barrier per stage.
__device__ __forceinline__ void base_sort(double* v, int* t, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size / 2; stride > 0; stride >>= 1) {
      const int i = threadIdx.x;
      if (i < n / 2) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = (lo & size) == 0;
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

// Entries of the sorted list (v, t)[0, n) ahead of (w, u).
__device__ __forceinline__ int base_rank_in(const double* v, const int* t, int n, double w, int u) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (base_before(v[mid], t[mid], w, u)) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// One block per expert.  Block 0 first advances the state.  A round that began
// with no unassigned token ends the phase: the final phase marks the auction
// done, an earlier one lowers eps and clears holders and assignments (every
// block takes its share).  Otherwise expert e collects its bidders in token
// order, at most kBaseCand (later ones stay unassigned and bid again), and
// ranks them and its holders in the order (bid desc, token asc) by counting;
// ranks below c are kept, holders ranked c or beyond are evicted.
__global__ __launch_bounds__(kBaseThreads) void base_resolve_kernel(BaseArgs a, int r) {
  const int e = blockIdx.x;
  const int tid = threadIdx.x;
  // every word the first decisions need, read together (one round trip)
  const int cnt = a.counts[r & 1], nbid = a.bid_cnt[e], nh = a.hold_n[e];
  const BaseState st = a.state[r & 1];
  const int n_un = st.done ? 0 : cnt;
  const bool fail = !st.done && n_un > 0 && st.rounds_phase >= a.max_rounds;
  if (e == 0 && tid == 0) {
    BaseState nx = st;
    if (!st.done) {
      if (n_un == 0) {
        if (st.eps <= st.eps_end) {
          nx.done = 1;
        } else {
          nx.eps = fmax(st.eps / kBaseEpsStep, st.eps_end);
          nx.phase = st.phase + 1;
          nx.rounds_phase = 0;
        }
      } else if (fail) {
        nx.done = 1;
        nx.failed = 1;
      } else {
        nx.rounds_phase = st.rounds_phase + 1;
        nx.rounds_total = st.rounds_total + 1;
      }
    }
    a.state[(r + 1) & 1] = nx;
    if (a.host_flag) {  // pacing for the host (synchronous form only)
      __hip_atomic_store(&a.host_flag->done, nx.done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      __hip_atomic_store(&a.host_flag->round, r, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
  if (st.done || fail) return;
  if (n_un == 0) {
    if (st.eps > st.eps_end) {  // next phase: prices kept
      if (tid == 0) a.hold_n[e] = 0;
      for (int64_t s = static_cast<int64_t>(e) * kBaseThreads + tid; s < a.S;
           s += static_cast<int64_t>(a.E) * kBaseThreads)
        a.assign[s] = -1;
    }
    return;
  }
  if (nbid == 0) return;

  extern __shared__ double base_lds[];
  const int c = a.cap;
  double* hv = base_lds;                             // holders [c]
  double* bv = hv + c;                               // bidders [kBaseCand]
  int* ht = reinterpret_cast<int*>(bv + kBaseCand);  // [c]
  int* bt = ht + c;                                  // [kBaseCand]
  __shared__ uint64_t masks[kBaseIters * kBaseWaves];
  __shared__ int offs[kBaseIters * kBaseWaves];
  __shared__ int pass_total;
  const int lane = lane_id(), w = tid / kWave;
  const int64_t base = static_cast<int64_t>(e) * c;
  for (int i = tid; i < nh; i += kBaseThreads) {
    hv[i] = a.hold_v[base + i];
    ht[i] = a.hold_t[base + i];
  }
  // bidders in token order: per pass kBaseIters tiles of kBaseThreads tokens;
  // a ballot mask per (tile, wave), an exclusive scan of their counts.  When
  // the expert takes all its bidders (at most kBaseCand) and the round has few,
  // they are found in the round's bidder list instead (in any order: the ranks
  // below use the total order alone, so the set decides the outcome).
  int have = 0;
  if (nbid <= kBaseCand && static_cast<int64_t>(n_un) * 8 <= a.S) {
    if (tid == 0) pass_total = 0;
    __syncthreads();
    for (int i0 = 0; i0 < n_un; i0 += 4 * kBaseThreads) {
      int t[4], be[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {  // unconditional loads (clamped), issued together
        const int i = i0 + q * kBaseThreads + tid;
        t[q] = a.blist[i < n_un ? i : 0];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) be[q] = a.bid_e[t[q]];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (i0 + q * kBaseThreads + tid < n_un && be[q] == e) {
          const int pos = atomicAdd(&pass_total, 1);  // < nbid <= kBaseCand
          if (pos < kBaseCand) bt[pos] = t[q];
        }
    }
    __syncthreads();
    have = min(pass_total, kBaseCand);  // == nbid
  } else
  for (int64_t p0 = 0; p0 < a.S && have < kBaseCand; p0 += static_cast<int64_t>(kBaseIters) * kBaseThreads) {
    int be[kBaseIters];
#pragma unroll
    for (int i = 0; i < kBaseIters; ++i) {  // unconditional loads (clamped), issued together
      const int64_t s = p0 + static_cast<int64_t>(i) * kBaseThreads + tid;
      be[i] = a.bid_e[s < a.S ? s : 0];
      if (s >= a.S) be[i] = -1;
    }
#pragma unroll
    for (int i = 0; i < kBaseIters; ++i) {
      const uint64_t m = __ballot(be[i] == e);
      if (lane == 0) masks[i * kBaseWaves + w] = m;
    }
    __syncthreads();
    if (w == 0) {  // exclusive scan of kBaseIters * kBaseWaves counts, 8 per lane
      constexpr int kPer = kBaseIters * kBaseWaves / kWave;
      int cnt[kPer], sum = 0;
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        cnt[j] = __popcll(masks[lane * kPer + j]);
        sum += cnt[j];
      }
      int incl = sum;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(incl, off, kWave);
        if (lane >= off) incl += y;
      }
      int run = incl - sum;
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        offs[lane * kPer + j] = run;
        run += cnt[j];
      }
      if (lane == kWave - 1) pass_total = incl;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kBaseIters; ++i) {
      if (be[i] == e) {
        const int k = i * kBaseWaves + w;
        const int pos = have + offs[k] + popc_below(masks[k]);
        if (pos < kBaseCand) bt[pos] = static_cast<int>(p0 + static_cast<int64_t>(i) * kBaseThreads + tid);
      }
    }
    have += pass_total;  // uniform
    __syncthreads();     // masks and offs are reused by the next pass
  }
  const int nb = min(have, kBaseCand);
  // the bids of the collected tokens, read together (bt is complete after the
  // last pass's barrier)
  for (int i = tid; i < nb; i += kBaseThreads) bv[i] = a.bid_v[bt[i]];
  __syncthreads();
  if (tid == 0) a.bid_cnt[e] = 0;  // for the next round (every thread has read it)
  if (nb > kBaseSortFrom) {
    // many bidders (the first rounds of a phase): sort them, then each entry's
    // rank in the union is its own index plus its rank in the other list
    int np2 = 1;
    while (np2 < nb) np2 <<= 1;
    for (int i = nb + tid; i < np2; i += kBaseThreads) {
      bv[i] = -INFINITY;
      bt[i] = 0x7fffffff;
    }
    __syncthreads();
    base_sort(bv, bt, np2);
    for (int i = tid; i < nh; i += kBaseThreads) {
      const double v = hv[i];
      const int t = ht[i];
      const int r_ = i + base_rank_in(bv, bt, nb, v, t);
      if (r_ < c) {
        a.hold_v[base + r_] = v;
        a.hold_t[base + r_] = t;
        if (r_ == c - 1) a.price[e] = v;
      } else {
        a.assign[t] = -1;  // evicted
      }
    }
    for (int j = tid; j < nb; j += kBaseThreads) {
      const double v = bv[j];
      const int t = bt[j];
      const int r_ = j + base_rank_in(hv, ht, nh, v, t);
      if (r_ < c) {
        a.hold_v[base + r_] = v;
        a.hold_t[base + r_] = t;
        a.assign[t] = e;
        if (r_ == c - 1) a.price[e] = v;
      }
    }
    if (tid == 0) {
      a.hold_n[e] = min(c, nh + nb);
      atomicAdd(&a.counts[2 + (r & 1)], min(c, nh + nb) - nh);
    }
    return;
  }
  // few bidders: ranks in the union of holders (sorted) and bidders (unsorted) by counting
  for (int i = tid; i < nh; i += kBaseThreads) {
    const double v = hv[i];
    const int t = ht[i];
    int r_ = i;
    for (int j = 0; j < nb; ++j) r_ += base_before(bv[j], bt[j], v, t);
    if (r_ < c) {
      a.hold_v[base + r_] = v;
      a.hold_t[base + r_] = t;
      if (r_ == c - 1) a.price[e] = v;
    } else {
      a.assign[t] = -1;  // evicted
    }
  }
  for (int j = tid; j < nb; j += kBaseThreads) {
    const double v = bv[j];
    const int t = bt[j];
    int r_ = 0;
    for (int q = 0; q < nb; ++q) r_ += base_before(bv[q], bt[q], v, t);
    int lo = 0, hi = nh;  // holders ahead of bidder j
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (base_before(hv[mid], ht[mid], v, t)) lo = mid + 1;
      else hi = mid;
    }
    r_ += lo;
    if (r_ < c) {
      a.hold_v[base + r_] = v;
      a.hold_t[base + r_] = t;
      a.assign[t] = e;
      if (r_ == c - 1) a.price[e] = v;
    }
  }
  if (tid == 0) {
    a.hold_n[e] = min(c, nh + nb);
    atomicAdd(&a.counts[2 + (r & 1)], min(c, nh + nb) - nh);
  }
}

// ---------------------------------------------------------------- one wave per bidder
// The bid of token t with the lanes over experts: the best value (lower expert
// on ties) and the best other value by butterflies over (value, expert); max
// is exact, so this equals the sequential scan of base_bid_kernel.  Every lane
// returns the same expert and bid.
// Token t's scores for experts q * 64 + lane, q < 4, loaded together (clamped:
// a lane past E reads expert 0).
__device__ __forceinline__ void base_row_load(const BaseArgs& a, int t, int lane, float (&lv)[4]) {
  const float* row = a.logits + static_cast<int64_t>(t) * a.E;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = q * kWave + lane;
    lv[q] = row[e < a.E ? e : 0];
  }
}

// base_wave_bid with the scores of the first 256 experts already loaded (lv0,
// from base_row_load).
__device__ __forceinline__ void base_wave_bid_from(const BaseArgs& a, const double* pr, double eps, int t, int lane,
                                                   const float (&lv0)[4], int& e_out, double& bid_out) {
  const float* row = a.logits + static_cast<int64_t>(t) * a.E;
  double v1 = -INFINITY, v2 = -INFINITY, l1 = 0.0;
  int e1 = 0x7fffffff;
  // four experts per lane per batch, loaded together past the first 256
  // (clamped: a lane past E reads expert 0 and skips it)
  for (int e0 = 0; e0 < a.E; e0 += 4 * kWave) {
    float lv[4];
    if (e0 == 0) {
#pragma unroll
      for (int q = 0; q < 4; ++q) lv[q] = lv0[q];
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = e0 + q * kWave + lane;
        lv[q] = row[e < a.E ? e : 0];
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = e0 + q * kWave + lane;
      if (e >= a.E) continue;
      const double v = static_cast<double>(lv[q]) - pr[e];
      if (v > v1) {
        v2 = v1;
        v1 = v;
        e1 = e;
        l1 = static_cast<double>(lv[q]);
      } else if (v > v2) {
        v2 = v;
      }
    }
  }
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const double ov1 = xor_partner(v1, off), ov2 = xor_partner(v2, off);
    const double ol1 = xor_partner(l1, off);
    const int oe1 = xor_partner(e1, off);
    if (ov1 > v1 || (ov1 == v1 && oe1 < e1)) {
      v2 = fmax(ov2, v1);
      v1 = ov1;
      e1 = oe1;
      l1 = ol1;
    } else {
      v2 = fmax(v2, ov1);
    }
  }
  if (a.E == 1) v2 = v1;
  e_out = e1;
  bid_out = l1 - v2 + eps;
}

__device__ __forceinline__ void base_wave_bid(const BaseArgs& a, const double* pr, double eps, int t, int lane,
                                              int& e_out, double& bid_out) {
  float lv[4];
  base_row_load(a, t, lane, lv);
  base_wave_bid_from(a, pr, eps, t, lane, lv, e_out, bid_out);
}

// Expert e takes the only bid for it this round, (bid, t): the holders ahead
// of it are counted by the lanes while staged in `hvs`/`hts` (LDS of c
// entries), then the holders behind it move up one place from there, the last
// one dropping out when the list is full.  Returns the evicted token or -1
// (and its scores in `next`, from base_row_load); `bad` is set if the bid does
// not rank below c (it always does: a bid exceeds its expert's price, the c-th
// best bid).
__device__ __forceinline__ int base_wave_place(const BaseArgs& a, double* pr, int* hn, int e, double bid, int t,
                                               int lane, double* hvs, int* hts, bool& bad, float (&next)[4]) {
  const int c = a.cap;
  const int nh = hn[e];
  const int64_t base = static_cast<int64_t>(e) * c;
  int p = 0, ev = -1;
  double vlast = 0.0;  // bid of the holder that ends at c - 1
  // holders read 8 per lane at a time, the loads of a batch issued together
  // (clamped: a slot past nh reads slot 0 and is skipped)
  for (int i0 = 0; i0 < nh; i0 += 8 * kWave) {
    double hv[8];
    int ht[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = i0 + q * kWave + lane;
      const int ic = i < nh ? i : 0;
      hv[q] = a.hold_v[base + ic];
      ht[q] = a.hold_t[base + ic];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = i0 + q * kWave + lane;
      if (i >= nh) continue;
      hvs[i] = hv[q];
      hts[i] = ht[q];
      p += base_before(hv[q], ht[q], bid, t);
      if (i == c - 1) ev = ht[q];
      if (i == c - 2) vlast = hv[q];
    }
  }
  p = group_reduce<kWave>(p, OpAdd());
  ev = group_reduce<kWave>(ev, OpMaxI());
  // the evictee bids next: its scores are requested now, so that their latency
  // overlaps the holder shift and the wait for its stores (unconditional: no
  // branch around loads)
  base_row_load(a, ev >= 0 ? ev : t, lane, next);
  vlast = __shfl(vlast, (c - 2) & (kWave - 1), kWave);
  bad = p >= c;
  if (bad) return -1;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  for (int i = p + lane; i < min(nh, c - 1); i += kWave) {
    a.hold_v[base + i + 1] = hvs[i];
    a.hold_t[base + i + 1] = hts[i];
  }
  if (lane == 0) {
    a.hold_v[base + p] = bid;
    a.hold_t[base + p] = t;
    a.assign[t] = e;
    if (ev >= 0) a.assign[ev] = -1;
    const int nn = min(c, nh + 1);
    if (nn == c) pr[e] = p == c - 1 ? bid : vlast;
    hn[e] = nn;
  }
  return ev;
}

// The holders of expert e and its bidders this round (lanes b < n with bit b of
// `bm` set: bids in bvv[b], tokens in U[b], kr[b] of them ahead of each one
// among themselves), ranked together: the holders are read once, top-down
// 8 x 64 at a time, and every holder and bidder goes straight to its rank in
// the union (a holder: its place plus the bidders ahead of it; a bidder: kr,
// or 0 without `kr`, plus the holders ahead of it); ranks below c are kept, the others join the
// unassigned list U2.  A batch is read whole before it is written and a
// holder only moves up, so no unread slot is overwritten.  One wave.
__device__ __forceinline__ void base_wave_merge(const BaseArgs& a, double* pr, int* hn, int e, uint64_t bm, int nbid,
                                            int n, const double* bvv, const int* U, const int* kr, int lane,
                                            int* U2, int* nU2) {
  const int c = a.cap;
  const bool mine = (bm >> lane) & 1;
  const uint2 lvb = __builtin_bit_cast(uint2, lane < n ? bvv[lane] : 0.0);
  const int lt = lane < n ? U[lane] : 0;
  int ahead_b = 0;  // lane b: holders ahead of bidder b
  const int nh = hn[e];
  const int64_t base = static_cast<int64_t>(e) * c;
  for (int hi = nh; hi > 0; hi -= 8 * kWave) {
    const int lo = max(0, hi - 8 * kWave);
    double hv[8];
    int ht[8], ahead[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = lo + q * kWave + lane;
      const int ic = i < hi ? i : lo;
      hv[q] = a.hold_v[base + ic];
      ht[q] = a.hold_t[base + ic];
      ahead[q] = 0;
    }
    for (uint64_t rem = bm; rem != 0; rem &= rem - 1) {  // uniform
      const int b = static_cast<int>(__builtin_ctzll(rem));
      const uint2 qb = {static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(lvb.x), b)),
                        static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(lvb.y), b))};
      const double bv = __builtin_bit_cast(double, qb);
      const int bt = __builtin_amdgcn_readlane(lt, b);
      int cnt = 0;  // holders of this batch ahead of bidder b
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (lo + q * kWave + lane >= hi) continue;
        const bool b_first = base_before(bv, bt, hv[q], ht[q]);
        ahead[q] += b_first;
        cnt += !b_first;
      }
      cnt = group_reduce<kWave>(cnt, OpAdd());
      if (lane == b) ahead_b += cnt;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = lo + q * kWave + lane;
      if (i >= hi) continue;
      const int nr = i + ahead[q];
      if (nr < c) {
        if (nr != i) {
          a.hold_v[base + nr] = hv[q];
          a.hold_t[base + nr] = ht[q];
        }
        if (nr == c - 1) pr[e] = hv[q];
      } else {
        a.assign[ht[q]] = -1;  // evicted
        const int pq = atomicAdd(nU2, 1);
        if (pq < kBaseTail) U2[pq] = ht[q];
      }
    }
  }
  // the expert's bidders at their ranks
  if (mine) {
    const int r = (kr ? kr[lane] : 0) + ahead_b;
    const double bv = __builtin_bit_cast(double, lvb);
    if (r < c) {
      a.hold_v[base + r] = bv;
      a.hold_t[base + r] = lt;
      a.assign[lt] = e;
      if (r == c - 1) pr[e] = bv;
    } else {
      const int pq = atomicAdd(nU2, 1);
      if (pq < kBaseTail) U2[pq] = lt;
    }
  }
  if (lane == 0) hn[e] = min(c, nh + nbid);
}

// The tail's unassigned lists: this round's and the next (filled by the
// merges) trade places; every thread swaps its own pointers after the barrier
// that completes the next list, and the count of the list that becomes the next
// one is cleared before its first append in the following round.
__device__ __forceinline__ void swap_lists(int*& U, int*& U2, int*& nU, int*& nU2) {
  int* t = U;
  U = U2;
  U2 = t;
  int* c = nU;
  nU = nU2;
  nU2 = c;
}

// ---------------------------------------------------------------- tail
// Most rounds of a phase have a handful of bidders.  Once at most kBaseTail
// tokens are unassigned after a round, one workgroup runs the following rounds
// itself, with the same arithmetic and the same rule (the union of holders and
// bidders ranked in the order (bid desc, token asc), ranks below c kept), until
// the phase has no unassigned token or more than kBaseTail of them; the next
// bid / resolve pair then carries on.  Prices and holder counts live in LDS
// meanwhile; holders stay sorted in device memory.  The order of the tokens in
// the unassigned list does not matter: every bid depends on its token alone and
// ranking uses a total order.
__global__ __launch_bounds__(kBaseThreads) void base_tail_kernel(BaseArgs a, int r) {
  BaseState* sp = a.state + ((r + 1) & 1);
  // unassigned after this round: those at its start less the slots its resolve
  // step filled; a round that began with none (and did not end the auction)
  // changed phase and unassigned all S.  The three words are read together,
  // before the first decision, so that a launch that has nothing to do waits
  // for one memory round trip.
  const int done = sp->done, un0 = a.counts[r & 1], filled = a.counts[2 + (r & 1)];
  if (done) return;
  const int64_t left = un0 > 0 ? un0 - filled : static_cast<int64_t>(a.S);
  if (left > kBaseTail) return;  // uniform: more than the tail takes
  const double eps = sp->eps;
  int rounds_phase = sp->rounds_phase, rounds_total = sp->rounds_total, failed = 0;
  extern __shared__ double tail_lds[];
  const int c = a.cap, E = a.E;
  double* pr = tail_lds;                              // prices [E]
  double* hvs = pr + E;                               // one expert's holder bids [c] (one-bidder rounds)
  int* hn = reinterpret_cast<int*>(hvs + c);          // holder counts [E]
  int* hts = hn + E;                                  // the holders' tokens [c]
  __shared__ int Ubuf[2][kBaseTail];  // unassigned tokens of this round and the next, swapped
  __shared__ int bex[kBaseTail], kr[kBaseTail], nbe[kBaseTail], ldr[kBaseTail];
  __shared__ double bvv[kBaseTail];
  __shared__ int nUbuf[2], nL, fast_rounds, fast_fail;
  const int tid = threadIdx.x, lane = lane_id(), w = tid / kWave;
  int* U = Ubuf[0];
  int* U2 = Ubuf[1];
  int* nU = &nUbuf[0];
  int* nU2 = &nUbuf[1];
  if (tid == 0) *nU = 0;
  __syncthreads();
  // unassigned tokens (any order)
  for (int64_t s0 = 0; s0 < a.S; s0 += 8 * kBaseThreads) {
    int v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {  // unconditional loads (clamped), issued together
      const int64_t s = s0 + q * kBaseThreads + tid;
      v[q] = a.assign[s < a.S ? s : 0];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
      if (v[q] < 0 && s0 + q * kBaseThreads + tid < a.S) {
        const int p = atomicAdd(nU, 1);
        if (p < kBaseTail) U[p] = static_cast<int>(s0 + q * kBaseThreads + tid);
      }
  }
  __syncthreads();
  if (*nU == 0 || *nU > kBaseTail) return;  // uniform
  for (int e = tid; e < E; e += kBaseThreads) {
    pr[e] = a.price[e];
    hn[e] = a.hold_n[e];
  }
  __syncthreads();
  for (;;) {
    const int n = *nU;  // uniform (read after a barrier)
    if (n == 0 || n > kBaseTail) break;
    if (rounds_phase >= a.max_rounds) {
      failed = 1;
      break;
    }
    if (n == 1) {
      // One bidder: it always wins a place (its bid exceeds its expert's
      // price, the c-th best bid) and pushes out at most one holder, who bids
      // next.  Wave 0 follows the chain: bid (lanes over experts, an exact
      // arg-max with the lower expert on ties and the best other value), the
      // holders ahead of it (lanes over holders, staged in LDS), then the
      // holders behind it move up by one.
      if (w == 0) {
        int t = U[0];
        int k = 0, fl = 0;
        float lv[4];
        base_row_load(a, t, lane, lv);
        for (;;) {
          if (rounds_phase + k >= a.max_rounds) {
            fl = 1;
            break;
          }
          int e1;
          double bid;
          base_wave_bid_from(a, pr, eps, t, lane, lv, e1, bid);
          bool bad;
          const int evicted = base_wave_place(a, pr, hn, e1, bid, t, lane, hvs, hts, bad, lv);
          if (bad) {  // cannot happen (see base_wave_place); stop rather than loop
            fl = 1;
            break;
          }
          ++k;
          // stores and LDS updates visible to the whole wave before the next step
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
          if (evicted < 0) {
            t = -1;
            break;
          }
          t = evicted;
        }
        if (lane == 0) {
          U[0] = t;
          *nU = t >= 0 ? 1 : 0;
          fast_rounds = k;
          fast_fail = fl;
        }
      }
      __syncthreads();
      rounds_phase += fast_rounds;
      rounds_total += fast_rounds;
      if (fast_fail) {
        failed = 1;
        break;
      }
      __syncthreads();  // fast_rounds and fast_fail are rewritten by a later chain
      continue;
    }
    // Up to 16 bidders: one wave each computes its bid; if they all want
    // different experts, each wave then places its own (one bid per expert),
    // else the general merge below runs on these bids.
    bool have_bids = false;
    if (n <= kBaseWaves) {
      if (w < n) {
        int e1;
        double bid;
        base_wave_bid(a, pr, eps, U[w], lane, e1, bid);
        if (lane == 0) {
          bex[w] = e1;
          bvv[w] = bid;
        }
      }
      if (tid == 0) {
        *nU2 = 0;
        fast_fail = 0;
      }
      __syncthreads();
      // distinct experts: each lane holds one bidder's expert (lanes past n a
      // sentinel of their own) and compares it with the others' by readlane
      bool distinct;
      {
        const int ei = lane < n ? bex[lane] : -1 - lane;
        bool clash = false;
#pragma unroll
        for (int j = 0; j < kBaseWaves; ++j) clash |= j != lane && __builtin_amdgcn_readlane(ei, j) == ei;
        distinct = __ballot(clash) == 0;
      }
      if (distinct) {  // uniform: every wave read the same bids
        if (w < n) base_wave_merge(a, pr, hn, bex[w], 1ull << w, 1, n, bvv, U, nullptr, lane, U2, nU2);
        __syncthreads();  // the next list and its count are complete
        swap_lists(U, U2, nU, nU2);
        rounds_phase += 1;
        rounds_total += 1;
        continue;
      }
      have_bids = true;
    }
    // bids of more than 16 bidders: 16 lanes each (up to 64 bidders)
    if (!have_bids) {
      const int g = tid / 16;
      if (g < n) {  // uniform in each group of 16 lanes
        int e1;
        double bid;
        base_group_bid<16>(a, pr, eps, U[g], tid % 16, e1, bid);
        if (tid % 16 == 0) {
          bex[g] = e1;
          bvv[g] = bid;
        }
      }
    }
    if (tid == 0) *nU2 = 0;
    __syncthreads();
    // 16 lanes per bidder: kr = bidders of the same expert ahead of it, nbe =
    // bidders of its expert; then wave 0 lists the best bidder of each expert
    // (kr == 0), which leads it
    {
      const int g = tid / 16, sub = tid % 16;
      int k = 0, m = 0;
      if (g < n) {
        const int e = bex[g];
        const double v = bvv[g];
        const int t = U[g];
        for (int j = sub; j < n; j += 16) {
          const bool same = bex[j] == e;
          m += same;
          k += same && base_before(bvv[j], U[j], v, t);
        }
      }
      k = group_reduce<16>(k, OpAdd());
      m = group_reduce<16>(m, OpAdd());
      if (g < n && sub == 0) {
        kr[g] = k;
        nbe[g] = m;
      }
    }
    __syncthreads();
    if (w == 0) {
      const bool lead = lane < n && kr[lane] == 0;
      const uint64_t lm = __ballot(lead);
      if (lead) ldr[popc_below(lm)] = lane;
      if (lane == 0) nL = __popcll(lm);
    }
    __syncthreads();
    // One wave per expert with bidders: its holders are read once, top-down
    // 8 x 64 at a time, and every holder and bidder of the expert goes straight
    // to its rank in the union (a holder: its place plus the expert's bidders
    // ahead of it; a bidder: kr plus the holders ahead of it); ranks below c
    // are kept.  A batch is read whole before it is written and a holder only
    // moves up, so no unread slot is overwritten.
    for (int li = w; li < nL; li += kBaseWaves) {
      const int e = bex[ldr[li]];
      const uint64_t bm = __ballot(lane < n && bex[lane] == e);
      base_wave_merge(a, pr, hn, e, bm, nbe[ldr[li]], n, bvv, U, kr, lane, U2, nU2);
    }
    __syncthreads();  // the next list and its count are complete
    swap_lists(U, U2, nU, nU2);
    rounds_phase += 1;
    rounds_total += 1;
  }
  for (int e = tid; e < E; e += kBaseThreads) {
    a.price[e] = pr[e];
    a.hold_n[e] = hn[e];
  }
  if (tid == 0) {
    sp->rounds_phase = rounds_phase;
    sp->rounds_total = rounds_total;
    if (failed) {
      sp->done = 1;
      sp->failed = 1;
    }
  }
}

// ---------------------------------------------------------------- outputs
// ids, weights (sigmoid of the score) and the wave-block histogram [E, nb]
// that the scan and assign kernels turn into slots
// With `status` (the asynchronous form) the outputs are written whatever the
// outcome, every token with a valid expert (its current one, else s mod E, so
// that the slot kernels that follow stay in bounds), and the outcome goes to
// status; without it (the host reads the state) only a finished auction writes.
__global__ __launch_bounds__(kBlock) void base_finish_kernel(BaseArgs a, int r, BaseDevStatus* status) {
  const BaseState st = a.state[r & 1];
  const bool ok = st.done && !st.failed;
  if (!ok && status == nullptr) return;
  extern __shared__ int hist_lds[];  // [kWavesPerBlock, E]
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = lane_id();
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kBlock + tid;
  const bool valid = s < a.S;
  if (status && blockIdx.x == 0 && tid == 0)
    *status = BaseDevStatus{st.phase + 1, st.rounds_total, st.eps, ok ? 0 : (st.failed == 2 ? 2 : 1), 0};
  int e = 0;
  if (valid) {
    e = a.assign[s];
    if (e < 0 || e >= a.E) e = static_cast<int>(s % a.E);
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
  if (a.prices_out && blockIdx.x == 0)
    for (int i = tid; i < a.E; i += kBlock) a.prices_out[i] = a.price[i];
}

// The outcome of an empty batch: nothing to assign.
__global__ void base_empty_status_kernel(BaseDevStatus* status) { *status = BaseDevStatus{0, 0, 0.0, 0, 0}; }

// ---------------------------------------------------------------- driver
size_t base_resolve_lds(int cap) { return static_cast<size_t>(cap + kBaseCand) * (sizeof(double) + sizeof(int)); }

// A pinned, device-mapped progress word per host thread (a synchronous call
// blocks its thread, so one suffices), allocated on first use and kept until
// the process ends; null if it cannot be had.
BaseHostFlag* base_host_flag() {
  thread_local BaseHostFlag* flag = nullptr;
  thread_local bool tried = false;
  if (!tried) {
    tried = true;
    void* p = nullptr;
    if (hipHostMalloc(&p, sizeof(BaseHostFlag), hipHostMallocMapped | hipHostMallocPortable) == hipSuccess)
      flag = static_cast<BaseHostFlag*>(p);
    else
      (void)hipGetLastError();  // clear the failure; pacing falls back to host reads
  }
  return flag;
}

hipError_t run_base_auction(const BaseArgs& a_in, hipStream_t st, BaseStats* stats) {
  hipError_t err;
  *stats = BaseStats{};
  if (a_in.S == 0) return hipSuccess;
  BaseArgs a = a_in;
  // HETUMOE_BASE_BATCHES=1 selects the batches (the path taken without pinned
  // memory), so that tests can compare the two
  const char* batches = getenv("HETUMOE_BASE_BATCHES");
  BaseHostFlag* hf = (batches && batches[0] == '1') ? nullptr : base_host_flag();
  a.host_flag = nullptr;
  if (hf) {
    void* dp = nullptr;
    if (hipHostGetDevicePointer(&dp, hf, 0) == hipSuccess) {
      a.host_flag = static_cast<BaseHostFlag*>(dp);
      __atomic_store_n(&hf->done, 0, __ATOMIC_RELAXED);
      __atomic_store_n(&hf->round, -1, __ATOMIC_RELEASE);
    } else {
      (void)hipGetLastError();
      hf = nullptr;
    }
  }
  const unsigned tok_blocks = static_cast<unsigned>((a.S + kBlock - 1) / kBlock);
  const size_t bid_lds = static_cast<size_t>(a.E) * (sizeof(double) + sizeof(int));
  const size_t tail_lds = static_cast<size_t>(a.E + a.cap) * (sizeof(double) + sizeof(int));
  const bool vec = a.E % 4 == 0 && reinterpret_cast<uintptr_t>(a.logits) % 16 == 0;
  base_range_kernel<<<kBaseRangeBlocks, kBaseThreads, 0, st>>>(a);
  base_init_kernel<<<1, kBaseRangeBlocks, 0, st>>>(a);
  base_reset_kernel<<<tok_blocks, kBlock, 0, st>>>(a);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  auto round = [&](int r) {
    if (vec) base_bid_kernel<true><<<tok_blocks, kBlock, bid_lds, st>>>(a, r);
    else base_bid_kernel<false><<<tok_blocks, kBlock, bid_lds, st>>>(a, r);
    base_resolve_kernel<<<static_cast<unsigned>(a.E), kBaseThreads, base_resolve_lds(a.cap), st>>>(a, r);
    base_tail_kernel<<<1, kBaseThreads, tail_lds, st>>>(a, r);
  };
  // the device ends the auction within (max_rounds + 1) rounds per phase; the
  // phases are at most 2 + log_32(2^30 / 4) < 8, so a bound of 12 phases is safe
  const int64_t limit = static_cast<int64_t>(a.max_rounds + 1) * 12 + 1;
  int r = 0;
  BaseState host{};
  if (hf) {
    // Paced: the host keeps kAhead rounds queued beyond the last one the device
    // has reached, and stops once the device reports the end.  A wait without
    // progress for a long time falls back to synchronizing the stream.
    constexpr int kAhead = 6;
    bool ended = false;
    for (; r < limit && !ended; ++r) {
      round(r);
      if ((err = hipGetLastError()) != hipSuccess) return err;
      if (r < kAhead) continue;
      const auto t0 = std::chrono::steady_clock::now();
      for (int spins = 0;; ++spins) {
        if (__atomic_load_n(&hf->done, __ATOMIC_ACQUIRE)) {
          ended = true;
          break;
        }
        if (__atomic_load_n(&hf->round, __ATOMIC_ACQUIRE) >= r - kAhead) break;
        if ((spins & 1023) == 1023 && std::chrono::steady_clock::now() - t0 > std::chrono::seconds(20)) {
          if ((err = hipStreamSynchronize(st)) != hipSuccess) return err;
          break;
        }
      }
    }
    if ((err = hipMemcpyAsync(&host, a.state + (r & 1), sizeof(host), hipMemcpyDeviceToHost, st)) != hipSuccess)
      return err;
    if ((err = hipStreamSynchronize(st)) != hipSuccess) return err;
    if (!host.done) host.failed = 1;  // the round limit: only a failing device gets here
  } else {
    int batch = 64;
    for (;;) {
      for (int i = 0; i < batch; ++i, ++r) round(r);
      if ((err = hipGetLastError()) != hipSuccess) return err;
      if ((err = hipMemcpyAsync(&host, a.state + (r & 1), sizeof(host), hipMemcpyDeviceToHost, st)) != hipSuccess)
        return err;
      if ((err = hipStreamSynchronize(st)) != hipSuccess) return err;
      if (host.done) break;
      if (r >= limit) {
        host.failed = 1;
        break;
      }
      batch = 128;
    }
  }
  stats->phases = host.phase + 1;
  stats->rounds = host.rounds_total;
  stats->eps = host.eps;
  stats->not_converged = host.failed == 1;
  stats->bad_scores = host.failed == 2;
  if (host.failed) return hipSuccess;
  base_finish_kernel<<<tok_blocks, kBlock, static_cast<size_t>(kWavesPerBlock) * a.E * sizeof(int), st>>>(a, r, nullptr);
  return hipGetLastError();
}

hipError_t run_base_auction_async(const BaseArgs& a, int launch_rounds, BaseDevStatus* status, hipStream_t st) {
  if (a.S == 0) {
    base_empty_status_kernel<<<1, 1, 0, st>>>(status);
    return hipGetLastError();
  }
  const unsigned tok_blocks = static_cast<unsigned>((a.S + kBlock - 1) / kBlock);
  const size_t bid_lds = static_cast<size_t>(a.E) * (sizeof(double) + sizeof(int));
  const size_t tail_lds = static_cast<size_t>(a.E + a.cap) * (sizeof(double) + sizeof(int));
  const bool vec = a.E % 4 == 0 && reinterpret_cast<uintptr_t>(a.logits) % 16 == 0;
  base_range_kernel<<<kBaseRangeBlocks, kBaseThreads, 0, st>>>(a);
  base_init_kernel<<<1, kBaseRangeBlocks, 0, st>>>(a);
  base_reset_kernel<<<tok_blocks, kBlock, 0, st>>>(a);
  for (int r = 0; r < launch_rounds; ++r) {
    if (vec) base_bid_kernel<true><<<tok_blocks, kBlock, bid_lds, st>>>(a, r);
    else base_bid_kernel<false><<<tok_blocks, kBlock, bid_lds, st>>>(a, r);
    base_resolve_kernel<<<static_cast<unsigned>(a.E), kBaseThreads, base_resolve_lds(a.cap), st>>>(a, r);
    base_tail_kernel<<<1, kBaseThreads, tail_lds, st>>>(a, r);
  }
  base_finish_kernel<<<tok_blocks, kBlock, static_cast<size_t>(kWavesPerBlock) * a.E * sizeof(int), st>>>(
      a, launch_rounds, status);
  return hipGetLastError();
}

}  // namespace hetumoe
