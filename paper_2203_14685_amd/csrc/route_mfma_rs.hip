// Register-stationary matrix-core route kernel: the bf16 logit projection x.W
// of Eq. 1 with softmax and expert selection (Sec. 3.1 top-k / kTop1), for
// shapes whose W fits in the register file of one CU.
//
// Persistent blocks of WAVES waves, one block per CU.  Each wave owns one K
// slice [sl*KSL, (sl+1)*KSL) of d = WAVES*KSL and keeps the B fragments of W^T
// for that slice (all E = 16*NT experts) in registers for the whole kernel, so
// W is read once per CU.  Eight waves (two per SIMD, up to 256 registers each)
// serve W up to 128 K elements.  The slices are dealt to the waves rotated by
// the block index, so that the blocks do not all read the same rows of W at
// the same moment; the partial sums are stored and added in slice order, so
// the result does not depend on the rotation.  Column n of N tile nt holds
// expert n*NT + nt, so a lane's NT experts are adjacent in a row of W and each
// K row of its fragments is one load.
// The block then streams 16-token tiles of x: each wave loads the tile's
// columns of its slice into one of two buffers while the other is multiplied
// (KSL/32 x NT v_mfma_f32_16x16x32_bf16), and the partial 16 x E tiles are
// summed in a fixed order through LDS.  K step ks of slice sl covers the columns
// [sl*KSL + 32ks, +32) and lane group g = lane/16 the 8 at sl*KSL + 32ks + 8g,
// so the 4 lanes of a row load 64 contiguous bytes per instruction.  The loads
// are unconditional (rows past the batch read its last row, results unused):
// a branch around them, or a register copy of a loaded value, would make the
// products wait for every load in flight.  After four tiles (one 64-token wave
// block) the block selects with WAVES lanes per token (each lane takes its
// E/WAVES logits from LDS at once, then a butterfly merge) and writes the wave block's
// (rank, expert) histogram.  The extended gates select here too: Dense-To-Sparse
// first turns the wave block's logits into (logits + noise) / temperature in
// LDS, and the hierarchical top-k (MODE 3) runs its two-level selection.
#include "select.hpp"

namespace hetumoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kGroupTokens = 64;  // one wave block
constexpr int kTileTokens = 16;   // MFMA M

// NT adjacent bf16 of one row of W (one load of NT * 2 bytes), as half-words.
template <int NT>
__device__ __forceinline__ void load_wrow(const uint16_t* p, uint16_t (&out)[NT]) {
  if constexpr (NT == 1) {
    out[0] = *p;
  } else if constexpr (NT == 2) {
    const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
    out[0] = static_cast<uint16_t>(v); out[1] = static_cast<uint16_t>(v >> 16);
  } else if constexpr (NT == 4) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    out[0] = static_cast<uint16_t>(v.x); out[1] = static_cast<uint16_t>(v.x >> 16);
    out[2] = static_cast<uint16_t>(v.y); out[3] = static_cast<uint16_t>(v.y >> 16);
  } else {
    static_assert(NT == 8, "NT in {1, 2, 4, 8}");
    const u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) { out[2 * i] = static_cast<uint16_t>(v[i]); out[2 * i + 1] = static_cast<uint16_t>(v[i] >> 16); }
  }
}

// MODE: 0 top-k, 1 kTop1, 3 hierarchical top-k
template <int WAVES, int NT, int KSL, int KMAX, int MODE>
__global__ __launch_bounds__(WAVES * 64) void route_mfma_rs_kernel(RouteArgs a) {
  constexpr int kThreads = WAVES * kWave;
  constexpr int E = NT * 16;
  constexpr int KSTEPS = KSL / 32;  // MFMA K steps per tile per wave
  constexpr int P = kThreads / kGroupTokens;  // selection lanes per token
  constexpr int SL = E / P;                   // logits per selection lane
  constexpr int LGS = E + 4;                  // row stride of lg: every lane's slice 16-byte aligned
  static_assert(KSTEPS * NT <= (WAVES == 8 ? 32 : 64), "W^T fragments must fit the register budget");
  static_assert(SL >= 2 && SL * P == E, "selection slices");
  __shared__ float part[WAVES * kTileTokens * E];      // per-slice partial logits of one tile
  __shared__ __align__(16) float lg[kGroupTokens * LGS];  // logits (+ bias) of the current wave block
  __shared__ int hist_lds[8 * E];                      // [k][E], k <= 8

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = lane_id();
  const int g = lane / 16, m = lane % 16;
  const int d = a.d;
  const int sl = (w + static_cast<int>(blockIdx.x)) % WAVES;  // K slice of this wave
  const int kbase = sl * KSL + 8 * g;  // + 32 ks per K step
  const uint16_t* wg = reinterpret_cast<const uint16_t*>(a.wg);
  const uint16_t* x = reinterpret_cast<const uint16_t*>(a.x);

  // W^T fragments of this lane: experts m*NT + nt, 8 consecutive K rows of
  // the slice per K step (one load per row, all issued before the packing)
  u32x4 bfr[KSTEPS][NT];
#pragma unroll
  for (int ks = 0; ks < KSTEPS; ++ks) {
    uint16_t r[8][NT];
#pragma unroll
    for (int j = 0; j < 8; ++j) load_wrow<NT>(wg + static_cast<int64_t>(kbase + 32 * ks + j) * E + m * NT, r[j]);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      uint32_t p[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) p[q] = static_cast<uint32_t>(r[2 * q][nt]) | (static_cast<uint32_t>(r[2 * q + 1][nt]) << 16);
      bfr[ks][nt] = u32x4{p[0], p[1], p[2], p[3]};
    }
  }

  // tiles of this block in order: wave block grp = blockIdx.x + (q / 4) * gridDim.x, tile q % 4
  const int nb = a.nb;
  const int my_groups = (nb - static_cast<int>(blockIdx.x) + static_cast<int>(gridDim.x) - 1) / static_cast<int>(gridDim.x);
  const int ntiles = 4 * my_groups;
  // the block's threads reduce expert tid % E of every row (kThreads is a
  // multiple of E); its bias is read once, not behind the x loads in flight
  const float bias_e = a.bias ? a.bias[tid % E] : 0.f;
  auto load_tile = [&](u32x4 (&buf)[KSTEPS], int q) {
    // rows past the batch, and the tile after the block's last, read the last
    // row of the batch: no branch around the loads, results never used
    const int64_t grp = blockIdx.x + static_cast<int64_t>(q / 4) * gridDim.x;
    int64_t row = grp * kGroupTokens + (q % 4) * kTileTokens + m;
    row = row < a.S ? row : a.S - 1;
    const u32x4* src = reinterpret_cast<const u32x4*>(x + row * d + kbase);
#pragma unroll
    for (int v = 0; v < KSTEPS; ++v) buf[v] = src[4 * v];
    __builtin_amdgcn_sched_barrier(0);  // the loads stay ahead of the products that follow
  };
  auto run_tile = [&](const u32x4 (&xt)[KSTEPS], int q) {
    const int t = q % 4;
    const int64_t grp = blockIdx.x + static_cast<int64_t>(q / 4) * gridDim.x;
    const int64_t tok0 = grp * kGroupTokens;
    if (t == 0)
      for (int i = tid; i < a.k * E; i += kThreads) hist_lds[i] = 0;
    f32x4 acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const bf16x8 av = __builtin_bit_cast(bf16x8, xt[ks]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bfr[ks][nt]), acc[nt], 0, 0, 0);
    }
    // partial tile of this wave's slice: lane holds rows 4g+i, experts m*NT + nt
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) part[(sl * kTileTokens + 4 * g + i) * E + m * NT + nt] = acc[nt][i];
    __syncthreads();
    for (int o = tid; o < kTileTokens * E; o += kThreads) {
      const int r = o / E, e = o % E;
      float sum = bias_e;
#pragma unroll
      for (int v = 0; v < WAVES; ++v) sum += part[(v * kTileTokens + r) * E + e];
      lg[(t * kTileTokens + r) * LGS + e] = sum;
    }
    __syncthreads();
    if (t != 3) return;

    // ------------------------------------------------ wave block complete
    if (a.temperature > 0.f) {
      // final logits of Dense-To-Sparse, in fp32 as the selection sees them
      for (int o = tid; o < kGroupTokens * E; o += kThreads) {
        const int r = o / E, e = o % E;
        if (tok0 + r < a.S) {
          float v = lg[r * LGS + e];
          if (a.noise) v += a.noise[(tok0 + r) * E + e];
          lg[r * LGS + e] = v / a.temperature;
        }
      }
      __syncthreads();
    }
    if (a.logits) {
      for (int o = tid; o < kGroupTokens * E; o += kThreads) {
        const int r = o / E, e = o % E;
        if (tok0 + r < a.S) a.logits[(tok0 + r) * E + e] = lg[r * LGS + e];
      }
    }
    const int tt = tid / P, j = tid % P;  // token of the wave block, lane within its P
    const int64_t s = tok0 + tt;
    const bool valid = s < a.S;
    if constexpr (MODE == 3)
      select_token_htopk_c<P, KMAX, SL>(&lg[tt * LGS], a.k, E / a.groups, a.normalize, j, valid, a.ids + s * a.k,
                                        a.weights + s * a.k, hist_lds);
    else
      select_token_c<P, KMAX, MODE == 1, SL>(&lg[tt * LGS], a.k, a.normalize, j, valid, a.ids + s * a.k,
                                             a.weights + s * a.k, hist_lds);
    __syncthreads();
    for (int i = tid; i < a.k * E; i += kThreads) {
      const int r = i / E, e = i % E;
      a.hist[(static_cast<int64_t>(r) * E + e) * nb + grp] = hist_lds[i];
    }
    __syncthreads();  // lg and hist_lds are reused by the next wave block
  };

  // two tile buffers in turn (the tile count is a multiple of 4): the next
  // tile's loads are in flight while the current one is multiplied
  u32x4 xa[KSTEPS], xb[KSTEPS];
  load_tile(xa, 0);
  for (int q = 0; q < ntiles; q += 2) {
    load_tile(xb, q + 1);
    run_tile(xa, q);
    load_tile(xa, q + 2);
    run_tile(xb, q + 1);
  }
}

// ---------------------------------------------------------------- launch
template <int WAVES, int NT, int KSL, int KMAX, int MODE>
static hipError_t launch_rs_t(const RouteArgs& a, int grid, hipStream_t st) {
  route_mfma_rs_kernel<WAVES, NT, KSL, KMAX, MODE><<<dim3(grid), dim3(WAVES * kWave), 0, st>>>(a);
  return hipGetLastError();
}

template <int WAVES, int NT, int KSL>
static hipError_t launch_rs_nt(const RouteArgs& a, int grid, hipStream_t st) {
  if (a.kind == 1) return launch_rs_t<WAVES, NT, KSL, 1, 1>(a, grid, st);
  // sorted lists no longer than k needs: each logit's insertion walks all of them
  if (a.kind == 3) {
    if (a.k == 1) return launch_rs_t<WAVES, NT, KSL, 1, 3>(a, grid, st);
    if (a.k == 2) return launch_rs_t<WAVES, NT, KSL, 2, 3>(a, grid, st);
    if (a.k <= 4) return launch_rs_t<WAVES, NT, KSL, 4, 3>(a, grid, st);
    return launch_rs_t<WAVES, NT, KSL, 8, 3>(a, grid, st);
  }
  if (a.k == 1) return launch_rs_t<WAVES, NT, KSL, 1, 0>(a, grid, st);
  if (a.k == 2) return launch_rs_t<WAVES, NT, KSL, 2, 0>(a, grid, st);
  if (a.k <= 4) return launch_rs_t<WAVES, NT, KSL, 4, 0>(a, grid, st);
  return launch_rs_t<WAVES, NT, KSL, 8, 0>(a, grid, st);
}

// Shapes served: bf16, E in {16, 32, 64, 128}, d in {512, 1024, 2048}, with
// d * E <= 131072, all with eight waves.
bool route_uses_mfma_rs(const RouteArgs& a) {
  if (a.kind == 2 || a.logits_in || a.dtype != 1) return false;
  if (a.E != 16 && a.E != 32 && a.E != 64 && a.E != 128) return false;
  if (a.d != 512 && a.d != 1024 && a.d != 2048) return false;
  if (static_cast<int64_t>(a.d) * a.E > 131072) return false;
  return (reinterpret_cast<uintptr_t>(a.x) % 16) == 0 && (reinterpret_cast<uintptr_t>(a.wg) % 16) == 0;
}

#ifndef HETUMOE_ROUTE_VALU_ONLY
bool route_fuses_extended(const RouteArgs& a) { return route_uses_mfma_rs(a); }
#else
bool route_fuses_extended(const RouteArgs&) { return false; }
#endif

hipError_t launch_route_mfma_rs(const RouteArgs& a, int cus, hipStream_t st) {
  const int grid = a.nb < cus ? a.nb : cus;
  const int key = a.E * 10000 + a.d;
  switch (key) {
    case 16 * 10000 + 512: return launch_rs_nt<8, 1, 64>(a, grid, st);
    case 16 * 10000 + 1024: return launch_rs_nt<8, 1, 128>(a, grid, st);
    case 16 * 10000 + 2048: return launch_rs_nt<8, 1, 256>(a, grid, st);
    case 32 * 10000 + 512: return launch_rs_nt<8, 2, 64>(a, grid, st);
    case 32 * 10000 + 1024: return launch_rs_nt<8, 2, 128>(a, grid, st);
    case 32 * 10000 + 2048: return launch_rs_nt<8, 2, 256>(a, grid, st);
    case 64 * 10000 + 512: return launch_rs_nt<8, 4, 64>(a, grid, st);
    case 64 * 10000 + 1024: return launch_rs_nt<8, 4, 128>(a, grid, st);
    case 64 * 10000 + 2048: return launch_rs_nt<8, 4, 256>(a, grid, st);
    case 128 * 10000 + 512: return launch_rs_nt<8, 8, 64>(a, grid, st);
    case 128 * 10000 + 1024: return launch_rs_nt<8, 8, 128>(a, grid, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hetumoe
