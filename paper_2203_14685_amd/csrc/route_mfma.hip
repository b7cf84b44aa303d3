// Route kernel on the matrix cores: the bf16 logit projection x.W of Eq. 1 on
// v_mfma_f32_16x16x32_bf16, with softmax and expert selection in the epilogue.
#include "select.hpp"

namespace hetumoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- MFMA route (bf16)
// 64 tokens per block, 4 waves; wave w computes the logits of tokens
// [16w, 16w+16) for all E = 16*NT experts with v_mfma_f32_16x16x32_bf16
// (M = tokens, N = experts, K = d).  Per K chunk of KC columns, W^T[:, kc:kc+KC]
// sits in LDS (B fragments are 16-byte LDS reads) and every lane holds 2*KC/4
// contiguous bytes of its token's row of x (A fragments).  The next chunk of
// both is loaded into registers while the current one is multiplied.  W [d, E]
// is transposed on the way: a thread loads an 8 x 8 block (8 rows of 8
// experts, 16 bytes each), regroups the half-words in registers and stores 8
// rows of W^T (8 columns each, 16 bytes).  Inside a
// chunk, lane group g = lane/16 supplies the columns [kc + (KC/4)*g,
// kc + (KC/4)*(g+1)); A and B use the same column order, so each MFMA sums a
// fixed permutation of 32 columns of the chunk.  The block's 64 x E logits
// (+ bias) then go to LDS and 4 lanes per token select.
constexpr int kMfmaTokens = 64;

template <int NT, int KC, int KMAX, bool KTOP1>
__global__ __launch_bounds__(kBlock) void route_mfma_kernel(RouteArgs a) {
  constexpr int E = NT * 16;
  constexpr int KG = KC / 4;                 // columns per lane group per chunk
  constexpr int KSTEPS = KG / 8;             // MFMAs per N tile per chunk
  constexpr int LDW = KC + 8;                // padded LDS row (bf16 elements) of W^T
  constexpr int WBLOCKS = (KC / 8) * (E / 8);  // 8 x 8 blocks of a W chunk
  constexpr int WVEC = (WBLOCKS + kBlock - 1) / kBlock;  // per thread
  constexpr int XVEC = KG / 8;               // 16-byte pieces of x per lane per chunk
  static_assert(E * LDW * 2 >= kMfmaTokens * (E + 1) * 4, "logits reuse the W^T buffer");
  __shared__ __align__(16) uint16_t wsT[E * LDW];
  __shared__ int hist_lds[8 * E];  // [k][E], k <= 8
  float* lg = reinterpret_cast<float*>(wsT);  // after the K loop: [64][E + 1] logits

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = lane_id();
  const int g = lane / 16, m = lane % 16;
  const int d = a.d;
  const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * kMfmaTokens;
  const int64_t arow = tok0 + w * 16 + m;  // token of this lane's A fragment rows
  const bool arow_ok = arow < a.S;
  const u32x4* xa = reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(a.x) + arow * d + KG * g);
  const uint16_t* wg = reinterpret_cast<const uint16_t*>(a.wg);

  f32x4 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 xcur[XVEC], xnxt[XVEC], wreg[WVEC][8];
  const u32x4 zero = {0u, 0u, 0u, 0u};
  // block b of a chunk: columns kb = 8 * (b / (E/8)) .. +8, experts eb = 8 * (b % (E/8)) .. +8
  auto load_w = [&](int kc0) {
#pragma unroll
    for (int v = 0; v < WVEC; ++v) {
      const int b = tid + v * kBlock;
      if (b < WBLOCKS) {
        const int kb = (b / (E / 8)) * 8, eb = (b % (E / 8)) * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          wreg[v][j] = *reinterpret_cast<const u32x4*>(wg + static_cast<int64_t>(kc0 + kb + j) * E + eb);
      }
    }
  };
#pragma unroll
  for (int v = 0; v < XVEC; ++v) xcur[v] = arow_ok ? xa[v] : zero;
  load_w(0);

  for (int kc = 0; kc < d; kc += KC) {
#pragma unroll
    for (int v = 0; v < WVEC; ++v) {
      const int b = tid + v * kBlock;
      if (b < WBLOCKS) {
        const int kb = (b / (E / 8)) * 8, eb = (b % (E / 8)) * 8;
        u32x4 col[8];
        transpose8x8_b16(wreg[v], col);
#pragma unroll
        for (int i = 0; i < 8; ++i) *reinterpret_cast<u32x4*>(&wsT[(eb + i) * LDW + kb]) = col[i];
      }
    }
    __syncthreads();
    const bool more = kc + KC < d;
    if (more) load_w(kc + KC);
#pragma unroll
    for (int v = 0; v < XVEC; ++v) xnxt[v] = (arow_ok && more) ? xa[(kc + KC) / 8 + v] : zero;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const bf16x8 av = __builtin_bit_cast(bf16x8, xcur[ks]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const u32x4 braw = *reinterpret_cast<const u32x4*>(&wsT[(nt * 16 + m) * LDW + KG * g + 8 * ks]);
        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, braw), acc[nt], 0, 0, 0);
      }
    }
    __syncthreads();  // wsT consumed before it is overwritten
#pragma unroll
    for (int v = 0; v < XVEC; ++v) xcur[v] = xnxt[v];
  }

  // logits (+ bias) of the block's 64 tokens into LDS: lane holds rows 4g+i of
  // the wave's 16 tokens, column m of each N tile
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int e = nt * 16 + m;
    const float b = a.bias ? a.bias[e] : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) lg[(w * 16 + 4 * g + i) * (E + 1) + e] = acc[nt][i] + b;
  }
  __syncthreads();
  if (a.logits) {
    for (int t = tid; t < kMfmaTokens * E; t += kBlock) {
      const int r = t / E, e = t % E;
      if (tok0 + r < a.S) a.logits[(tok0 + r) * E + e] = lg[r * (E + 1) + e];
    }
  }
  // selection: 4 lanes per token; (rank, expert) counts in LDS
  for (int i = tid; i < a.k * E; i += kBlock) hist_lds[i] = 0;
  __syncthreads();
  {
    const int tt = tid / 4, j = tid % 4;
    const int64_t s = tok0 + tt;
    select_token<4, KMAX, KTOP1>(&lg[tt * (E + 1)], E, a.k, a.normalize, j, s < a.S, a.ids + s * a.k,
                                 a.weights + s * a.k, hist_lds);
  }
  __syncthreads();
  for (int i = tid; i < a.k * E; i += kBlock) {
    const int r = i / E, e = i % E;
    a.hist[(static_cast<int64_t>(r) * E + e) * a.nb + blockIdx.x] = hist_lds[i];
  }
}

template <int NT, int KC, int KMAX, bool KTOP1>
static hipError_t launch_mfma_t(const RouteArgs& a, hipStream_t st) {
  route_mfma_kernel<NT, KC, KMAX, KTOP1><<<dim3(a.nb), dim3(kBlock), 0, st>>>(a);
  return hipGetLastError();
}

template <int NT, int KC>
static hipError_t launch_mfma_nt(const RouteArgs& a, hipStream_t st) {
  if (a.kind == 1) return launch_mfma_t<NT, KC, 1, true>(a, st);
  if (a.k == 1) return launch_mfma_t<NT, KC, 1, false>(a, st);
  if (a.k == 2) return launch_mfma_t<NT, KC, 2, false>(a, st);
  if (a.k <= 4) return launch_mfma_t<NT, KC, 4, false>(a, st);
  return launch_mfma_t<NT, KC, 8, false>(a, st);
}

bool route_uses_mfma(const RouteArgs& a) {
  return a.kind != 2 && !a.logits_in && a.dtype == 1 && a.E % 16 == 0 && a.E <= 128 &&
         a.d % (a.E <= 64 ? 256 : 128) == 0 && (reinterpret_cast<uintptr_t>(a.wg) % 16) == 0;
}

hipError_t launch_route_mfma(const RouteArgs& a, hipStream_t st) {
  switch (a.E / 16) {
    case 1: return launch_mfma_nt<1, 256>(a, st);
    case 2: return launch_mfma_nt<2, 256>(a, st);
    case 3: return launch_mfma_nt<3, 256>(a, st);
    case 4: return launch_mfma_nt<4, 256>(a, st);
    case 5: return launch_mfma_nt<5, 128>(a, st);
    case 6: return launch_mfma_nt<6, 128>(a, st);
    case 7: return launch_mfma_nt<7, 128>(a, st);
    default: return launch_mfma_nt<8, 128>(a, st);
  }
}

}  // namespace hetumoe
