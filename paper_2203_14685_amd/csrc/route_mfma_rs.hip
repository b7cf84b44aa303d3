// Register-stationary matrix-core route kernel: the bf16 logit projection x.W
// of Eq. 1 with softmax and expert selection (Sec. 3.1 top-k / kTop1), for
// shapes whose W fits in the register file of one CU.
//
// Persistent blocks of 8 waves, one per CU.  Wave w owns the K slice
// [w*KSL, (w+1)*KSL) of d = 8*KSL and keeps the B fragments of W^T for that
// slice (all E = 16*NT experts) in registers for the whole kernel, so W is read
// once per CU.  The block then streams 16-token tiles of x: each wave loads the
// tile's columns of its slice (one tile ahead), runs KSL/32 x NT
// v_mfma_f32_16x16x32_bf16, and the 8 partial 16 x E tiles are summed in a
// fixed order through LDS.  K step ks of wave w covers the columns
// [w*KSL + 32ks, +32) and lane group g = lane/16 the 8 at w*KSL + 32ks + 8g, so
// the 4 lanes of a row load 64 contiguous bytes per instruction.
// After four tiles (one 64-token wave block) the block selects with 8 lanes
// per token (each lane streams E/8 experts, then a butterfly merge) and writes
// the wave block's (rank, expert) histogram.
#include "select.hpp"

namespace hetumoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kRsWaves = 8;
constexpr int kRsThreads = kRsWaves * kWave;
constexpr int kGroupTokens = 64;  // one wave block
constexpr int kTileTokens = 16;   // MFMA M

template <int NT, int KSL, int KMAX, bool KTOP1>
__global__ __launch_bounds__(kRsThreads) void route_mfma_rs_kernel(RouteArgs a) {
  constexpr int E = NT * 16;
  constexpr int KSTEPS = KSL / 32;  // MFMA K steps per tile per wave
  static_assert(KSTEPS * NT <= 16, "W^T fragments must fit the register budget");
  __shared__ float part[kRsWaves * kTileTokens * E];   // per-wave partial logits of one tile
  __shared__ float lg[kGroupTokens * (E + 1)];         // logits (+ bias) of the current wave block
  __shared__ int hist_lds[8 * E];                      // [k][E], k <= 8

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = lane_id();
  const int g = lane / 16, m = lane % 16;
  const int d = a.d;
  const int kbase = w * KSL + 8 * g;  // + 32 ks per K step
  const uint16_t* wg = reinterpret_cast<const uint16_t*>(a.wg);
  const uint16_t* x = reinterpret_cast<const uint16_t*>(a.x);

  // W^T fragments of this lane: column m of each N tile, 8 consecutive columns
  // of the slice per K step
  u32x4 bfr[KSTEPS][NT];
#pragma unroll
  for (int ks = 0; ks < KSTEPS; ++ks) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const uint16_t* col = wg + static_cast<int64_t>(kbase + 32 * ks) * E + nt * 16 + m;
      uint32_t p[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        p[q] = static_cast<uint32_t>(col[(2 * q) * E]) | (static_cast<uint32_t>(col[(2 * q + 1) * E]) << 16);
      bfr[ks][nt] = u32x4{p[0], p[1], p[2], p[3]};
    }
  }

  // tiles of this block in order: wave block grp = blockIdx.x + (q / 4) * gridDim.x, tile q % 4
  const int nb = a.nb;
  const int my_groups = (nb - static_cast<int>(blockIdx.x) + static_cast<int>(gridDim.x) - 1) / static_cast<int>(gridDim.x);
  const int ntiles = 4 * my_groups;
  const u32x4 zero = {0u, 0u, 0u, 0u};
  auto tile_row = [&](int q) -> int64_t {
    const int64_t grp = blockIdx.x + static_cast<int64_t>(q / 4) * gridDim.x;
    return grp * kGroupTokens + (q % 4) * kTileTokens + m;
  };
  u32x4 xcur[KSTEPS], xnxt[KSTEPS];
  {
    const int64_t row = tile_row(0);
    const u32x4* src = reinterpret_cast<const u32x4*>(x + row * d + kbase);
#pragma unroll
    for (int v = 0; v < KSTEPS; ++v) xcur[v] = (ntiles > 0 && row < a.S) ? src[4 * v] : zero;
  }

  for (int q = 0; q < ntiles; ++q) {
    const int t = q % 4;
    const int64_t grp = blockIdx.x + static_cast<int64_t>(q / 4) * gridDim.x;
    const int64_t tok0 = grp * kGroupTokens;
    if (t == 0)
      for (int i = tid; i < a.k * E; i += kRsThreads) hist_lds[i] = 0;
    // prefetch the next tile
    {
      const int64_t row = tile_row(q + 1);
      const u32x4* src = reinterpret_cast<const u32x4*>(x + row * d + kbase);
      const bool ok = q + 1 < ntiles && row < a.S;
#pragma unroll
      for (int v = 0; v < KSTEPS; ++v) xnxt[v] = ok ? src[4 * v] : zero;
    }
    f32x4 acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const bf16x8 av = __builtin_bit_cast(bf16x8, xcur[ks]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bfr[ks][nt]), acc[nt], 0, 0, 0);
    }
    // partial tile of this wave: lane holds rows 4g+i, column m of each N tile
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) part[(w * kTileTokens + 4 * g + i) * E + nt * 16 + m] = acc[nt][i];
    __syncthreads();
    for (int o = tid; o < kTileTokens * E; o += kRsThreads) {
      const int r = o / E, e = o % E;
      float sum = a.bias ? a.bias[e] : 0.f;
#pragma unroll
      for (int v = 0; v < kRsWaves; ++v) sum += part[(v * kTileTokens + r) * E + e];
      lg[(t * kTileTokens + r) * (E + 1) + e] = sum;
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < KSTEPS; ++v) xcur[v] = xnxt[v];
    if (t != 3) continue;

    // ------------------------------------------------ wave block complete
    if (a.logits) {
      for (int o = tid; o < kGroupTokens * E; o += kRsThreads) {
        const int r = o / E, e = o % E;
        if (tok0 + r < a.S) a.logits[(tok0 + r) * E + e] = lg[r * (E + 1) + e];
      }
    }
    const int tt = tid / 8, j = tid % 8;  // token of the wave block, lane within its 8
    const int64_t s = tok0 + tt;
    const bool valid = s < a.S;
    select_token<8, KMAX, KTOP1>(&lg[tt * (E + 1)], E, a.k, a.normalize, j, valid, a.ids + s * a.k,
                                 a.weights + s * a.k, hist_lds);
    __syncthreads();
    for (int i = tid; i < a.k * E; i += kRsThreads) {
      const int r = i / E, e = i % E;
      a.hist[(static_cast<int64_t>(r) * E + e) * nb + grp] = hist_lds[i];
    }
    __syncthreads();  // lg and hist_lds are reused by the next wave block
  }
}

// ---------------------------------------------------------------- launch
template <int NT, int KSL, int KMAX, bool KTOP1>
static hipError_t launch_rs_t(const RouteArgs& a, int grid, hipStream_t st) {
  route_mfma_rs_kernel<NT, KSL, KMAX, KTOP1><<<dim3(grid), dim3(kRsThreads), 0, st>>>(a);
  return hipGetLastError();
}

template <int NT, int KSL>
static hipError_t launch_rs_nt(const RouteArgs& a, int grid, hipStream_t st) {
  if (a.kind == 1) return launch_rs_t<NT, KSL, 1, true>(a, grid, st);
  if (a.k == 1) return launch_rs_t<NT, KSL, 1, false>(a, grid, st);
  if (a.k == 2) return launch_rs_t<NT, KSL, 2, false>(a, grid, st);
  return launch_rs_t<NT, KSL, 8, false>(a, grid, st);
}

// Shapes served: bf16, E in {16, 32, 64, 128}, d in {512, 1024, 2048}, with the
// W^T fragments of a slice within 64 registers (d * E <= 65536); larger W spill.
bool route_uses_mfma_rs(const RouteArgs& a) {
  if (a.kind == 2 || a.logits_in || a.dtype != 1) return false;
  if (a.E != 16 && a.E != 32 && a.E != 64 && a.E != 128) return false;
  if (a.d != 512 && a.d != 1024 && a.d != 2048) return false;
  if (static_cast<int64_t>(a.d) * a.E > 65536) return false;
  return (reinterpret_cast<uintptr_t>(a.x) % 16) == 0;
}

hipError_t launch_route_mfma_rs(const RouteArgs& a, int cus, hipStream_t st) {
  const int grid = a.nb < cus ? a.nb : cus;
  const int key = a.E * 10000 + a.d;
  switch (key) {
    case 16 * 10000 + 512: return launch_rs_nt<1, 64>(a, grid, st);
    case 16 * 10000 + 1024: return launch_rs_nt<1, 128>(a, grid, st);
    case 16 * 10000 + 2048: return launch_rs_nt<1, 256>(a, grid, st);
    case 32 * 10000 + 512: return launch_rs_nt<2, 64>(a, grid, st);
    case 32 * 10000 + 1024: return launch_rs_nt<2, 128>(a, grid, st);
    case 32 * 10000 + 2048: return launch_rs_nt<2, 256>(a, grid, st);
    case 64 * 10000 + 512: return launch_rs_nt<4, 64>(a, grid, st);
    case 64 * 10000 + 1024: return launch_rs_nt<4, 128>(a, grid, st);
    case 128 * 10000 + 512: return launch_rs_nt<8, 64>(a, grid, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hetumoe
