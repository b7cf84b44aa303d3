// Gradient of the gate (step 1 of Algorithm 1, Eq. 1) for end-to-end training:
// dL from dw through the softmax of Eq. 1 (or its Switch / kTop1 readings) and
// the load-balancing loss, then dW = x^T dL, db = column sums of dL and
// dx = dL W^T.  Sums over tokens run in fixed ranges and a fixed order, so the
// results are bitwise reproducible; there are no atomics on floats.
//
// bf16 shapes with E a multiple of 16 (up to 128) and d a multiple of 64 run
// the two products on the matrix cores (v_mfma_f32_16x16x32_bf16).  x and W
// are exact in bf16; dL is fp32, so it is split into three bf16 parts whose sum
// is dL exactly and each part is multiplied separately: every product is then
// exact and only the fp32 accumulation rounds, as on the vector path.
#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kBwdWaves = 4;
constexpr int kBwdThreads = kBwdWaves * kWave;

template <int P>
__device__ __forceinline__ float group_max(float v) {
  return group_reduce<P>(v, OpMaxF());
}

template <int P>
__device__ __forceinline__ float group_sum(float v) {
  return group_reduce<P>(v, OpAdd());
}

// Sum over the lanes that hold the same position within their group of P, i.e.
// over lanes l, l + P, l + 2P, ... (the butterfly steps M = P .. 32).
template <int P>
__device__ __forceinline__ float across_groups_sum(float v) {
  if constexpr (P <= 1) v = xor_step<1>(v, OpAdd());
  if constexpr (P <= 2) v = xor_step<2>(v, OpAdd());
  if constexpr (P <= 4) v = xor_step<4>(v, OpAdd());
  if constexpr (P <= 8) v = xor_step<8>(v, OpAdd());
  if constexpr (P <= 16) v = xor_step<16>(v, OpAdd());
  if constexpr (P <= 32) v = xor_step<32>(v, OpAdd());
  return v;
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// v = hi + mid + lo with three bf16 parts (each remainder is exact in fp32).
__device__ __forceinline__ void split3(float v, uint32_t& h, uint32_t& m, uint32_t& l) {
  h = f32_to_bf16_bits(v);
  const float r1 = v - bf16_bits_to_f32(h);
  m = f32_to_bf16_bits(r1);
  const float r2 = r1 - bf16_bits_to_f32(m);
  l = f32_to_bf16_bits(r2);
}

__device__ __forceinline__ void split8(const float (&v)[8], u32x4& hi, u32x4& mi, u32x4& lo) {
  uint32_t h[8], m[8], l[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) split3(v[q], h[q], m[q], l[q]);
  hi = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
  mi = u32x4{m[0] | (m[1] << 16), m[2] | (m[3] << 16), m[4] | (m[5] << 16), m[6] | (m[7] << 16)};
  lo = u32x4{l[0] | (l[1] << 16), l[2] | (l[3] << 16), l[4] | (l[5] << 16), l[6] | (l[7] << 16)};
}

__device__ __forceinline__ f32x4 mfma_bf16(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

// ---------------------------------------------------------------- column sums
// out[e] = sum over rows b of part[b][e]: 16 threads per column take rows
// q, q + 16, ... in order, then their 16 sums are added in order.
// Column sums of part [rows, E] for the 64 columns of column block cb, 16
// threads per column (1024 threads): 8 rows' loads in flight, added in row
// order, then the 16 partial sums in order.  Returns the total on the threads
// of the first wave (q == 0) and writes it to out[e].
template <typename T>
__device__ __forceinline__ T colsum_cols(const T* part, int64_t rows, int E, T* out, int cb, T (*red)[kWave]) {
  const int q = threadIdx.x / kWave, c = threadIdx.x % kWave;
  const int e = cb * kWave + c;
  T v = 0;
  if (e < E) {
    for (int64_t b0 = q; b0 < rows; b0 += 16 * 8) {
      T t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int64_t b = b0 + 16 * u;
        t[u] = b < rows ? part[b * E + e] : T(0);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) v += t[u];
    }
  }
  red[q][c] = v;
  __syncthreads();
  T t = 0;
  if (q == 0 && e < E) {
    for (int i = 0; i < 16; ++i) t += red[i][c];
    out[e] = t;
  }
  return t;
}

template <typename T>
__global__ __launch_bounds__(1024) void colsum_kernel(const T* part, int64_t rows, int E, T* out) {
  __shared__ T red[16][kWave];
  colsum_cols(part, rows, E, out, blockIdx.x, red);
}

// ---------------------------------------------------------------- first choices
// Per block of kCountTokens tokens: counts of first choices per expert (integer
// atomics in LDS; counts do not depend on the order).
constexpr int kCountTokens = 4096;

__global__ __launch_bounds__(1024) void aux_counts_kernel(GateBwdArgs a, int32_t* cpart) {
  extern __shared__ int h[];
  for (int e = threadIdx.x; e < a.E; e += blockDim.x) h[e] = 0;
  __syncthreads();
  const int64_t s0 = static_cast<int64_t>(blockIdx.x) * kCountTokens;
  const int64_t s1 = min(static_cast<int64_t>(a.S), s0 + kCountTokens);
  for (int64_t s = s0 + threadIdx.x; s < s1; s += blockDim.x) {
    const int e = a.ids[s * a.k];
    if (e >= 0 && e < a.E) atomicAdd(&h[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < a.E; e += blockDim.x) cpart[static_cast<int64_t>(blockIdx.x) * a.E + e] = h[e];
}

// With at most kCountRowsInline rows of partial counts there is no column-sum
// launch: the dL blocks stage the rows in LDS and add them up themselves, as
// do the loss kernels (integer sums: exact in any order).
constexpr int kCountRowsInline = 16;

__host__ __device__ inline int count_rows(int S) { return (S + kCountTokens - 1) / kCountTokens; }

// First-choice count of expert e for the loss kernels.
__device__ __forceinline__ int first_count(const GateBwdArgs& a, int e) {
  const int rows = count_rows(a.S);
  if (rows > kCountRowsInline) return a.cnt[e];
  const int32_t* cpart = a.cnt + a.E;
  int c = 0;
  for (int r = 0; r < rows; ++r) c += cpart[static_cast<int64_t>(r) * a.E + e];
  return c;
}

// ---------------------------------------------------------------- dL
// One block per 64-token wave block of WAVES waves, each taking 64 / WAVES
// tokens.  P lanes per token (a power of two, 4 <= P <= 64), EPL experts per
// lane: lane j of a token holds experts j, j + P, ...  Softmax maxima and sums
// are butterfly reductions over the P lanes.  Also per wave block: sums of dL
// (for db) and of the softmax (load-balancing loss), and, for the matrix-core
// dW, dL transposed and split into three bf16 planes.
template <int P, int EPL, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void gate_dl_kernel(GateBwdArgs a) {
  constexpr int TP = kWave / P;                  // tokens per pass
  constexpr int TW = kWave / WAVES;              // tokens per wave
  constexpr int PASSES = TW / TP;
  static_assert(TW % TP == 0, "whole passes");
  extern __shared__ float sh[];  // [64][E + 1] dL tile (dlt only), then [2][WAVES][E] sums;
                                 // the partial counts after the larger of the two
  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
  const int j = lane % P, sub = lane / P;
  const int64_t wb = blockIdx.x;
  const int E = a.E, k = a.k;
  const bool aux = a.aux_coef != 0.f;
  const bool topk = a.kind != 1;  // top-k and hierarchical top-k share the weights
  const bool full_softmax = topk && (a.normalize == 0 || aux);
  const float inv_s = a.S > 0 ? 1.f / static_cast<float>(a.S) : 0.f;
  const float c_aux = a.aux_coef * static_cast<float>(E) * inv_s;
  // first-choice counts: cnt, or the partial rows added up here (below)
  const int crows = aux && count_rows(a.S) <= kCountRowsInline ? count_rows(a.S) : 0;
  float f[EPL], psum[EPL], bsum[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = j + P * i;
    f[i] = (aux && crows == 0 && e < E) ? static_cast<float>(a.cnt[e]) * inv_s : 0.f;
    psum[i] = 0.f;
    bsum[i] = 0.f;
  }

  for (int pass = 0; pass < PASSES; ++pass) {
    const int tok = TW * w + pass * TP + sub;
    const int64_t s = wb * kWave + tok;
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
    // chosen experts and their gradients, loaded together (out-of-range ids
    // are ignored); the chosen logits come from the token's own lanes: expert
    // e is element e / P of lane e % P of the token
    int idr[8];
    float dwr[8], lr[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      int e = -1;
      float g = 0.f;
      if (r < k) {
        const int64_t q = (valid ? s : 0) * k + r;
        e = a.ids[q];
        g = a.dw[q];
      }
      const bool ok = valid && e >= 0 && e < E;
      idr[r] = ok ? e : -1;
      dwr[r] = ok ? g : 0.f;
    }
    if (pass == 0 && crows > 0) {
      // the partial counts, one load per thread, issued after this pass's
      // logits so that the two latencies overlap; staged past the tile and
      // the sums, so nothing overwrites them
      int* cs = reinterpret_cast<int*>(sh + max(a.dlt ? kWave * (E + 1) : 0, 2 * WAVES * E));
      const int32_t* cpart = a.cnt + E;
      for (int q = threadIdx.x; q < crows * E; q += WAVES * kWave) cs[q] = cpart[q];
      __syncthreads();
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const int e = j + P * i;
        if (e >= E) continue;
        int c = 0;
        for (int r = 0; r < crows; ++r) c += cs[r * E + e];
        f[i] = static_cast<float>(c) * inv_s;
      }
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      lr[r] = -INFINITY;
      if (r < k) {
        const int e = idr[r] >= 0 ? idr[r] : 0;
        float cand = v[0];
#pragma unroll
        for (int i = 1; i < EPL; ++i)
          if (e / P == i) cand = v[i];
        const float got = __shfl(cand, (lane & ~(P - 1)) | (e % P), kWave);
        lr[r] = idr[r] >= 0 ? got : -INFINITY;
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
    if (topk && a.normalize) {
      // softmax over the k chosen logits
      float m2 = -INFINITY;
#pragma unroll
      for (int r = 0; r < 8; ++r) m2 = fmaxf(m2, lr[r]);
      float den = 0.f, wr[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        wr[r] = idr[r] >= 0 ? expf(lr[r] - m2) : 0.f;
        den += wr[r];
      }
      float inner = 0.f;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        wr[r] = idr[r] >= 0 ? wr[r] / den : 0.f;
        inner += wr[r] * dwr[r];
      }
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        if (idr[r] < 0) continue;
        const float gr = wr[r] * (dwr[r] - inner);
#pragma unroll
        for (int i = 0; i < EPL; ++i)
          if (j + P * i == idr[r]) dl[i] += gr;
      }
    } else if (topk) {
      // full softmax read at each chosen expert
      float gsum = 0.f;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        if (idr[r] < 0) continue;
        const float t = dwr[r] * (expf(lr[r] - m) / se);
        gsum += t;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
          if (j + P * i == idr[r]) dl[i] += t;
      }
#pragma unroll
      for (int i = 0; i < EPL; ++i) dl[i] -= p[i] * gsum;
    } else if (EPL <= 8 && E == P * EPL && k == EPL) {
      // kTop1 with groups of exactly P experts: element i of every lane is
      // expert j + P i, which lies in group i, so the k groups' maxima and
      // sums reduce side by side (the same arithmetic as the loop below)
      float mg[EPL], sg[EPL];
#pragma unroll
      for (int i = 0; i < EPL; ++i) mg[i] = group_max<P>(v[i]);
#pragma unroll
      for (int i = 0; i < EPL; ++i) sg[i] = group_sum<P>(expf(v[i] - mg[i]));
#pragma unroll
      for (int i = 0; i < (EPL <= 8 ? EPL : 8); ++i) {
        const int lo = i * P, id = idr[i];
        if (id < lo || id >= lo + P) continue;
        const float scale = dwr[i] * (expf(lr[i] - mg[i]) / sg[i]);
        dl[i] += scale * ((j + P * i == id ? 1.f : 0.f) - expf(v[i] - mg[i]) / sg[i]);
      }
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
    if (a.temperature > 0.f) {
      // the logits were (L + noise) / temperature: chain rule to L
#pragma unroll
      for (int i = 0; i < EPL; ++i) dl[i] = dl[i] / a.temperature;
    }
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = j + P * i;
      if (e >= E) continue;
      if (valid) {
        a.dl[s * E + e] = dl[i];
        bsum[i] += dl[i];
      }
      if (a.dlt) sh[tok * (E + 1) + e] = valid ? dl[i] : 0.f;
    }
  }
  // sums over the token lanes of each wave
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    bsum[i] = across_groups_sum<P>(bsum[i]);
    psum[i] = across_groups_sum<P>(psum[i]);
  }
  __syncthreads();  // dL tile complete
  if (a.dlt) {
    // 8 consecutive tokens of one expert per thread: one 16-byte store per
    // plane (s_pad is a multiple of 64, so the pieces are 16-byte aligned)
    const int64_t plane = static_cast<int64_t>(E) * a.s_pad;
    for (int q = threadIdx.x; q < E * (kWave / 8); q += WAVES * kWave) {
      const int e = q / (kWave / 8), t0 = (q % (kWave / 8)) * 8;
      float v8[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v8[u] = sh[(t0 + u) * (E + 1) + e];
      u32x4 hi, mi, lo;
      split8(v8, hi, mi, lo);
      const int64_t o = static_cast<int64_t>(e) * a.s_pad + wb * kWave + t0;
      *reinterpret_cast<u32x4*>(a.dlt + o) = hi;
      *reinterpret_cast<u32x4*>(a.dlt + plane + o) = mi;
      *reinterpret_cast<u32x4*>(a.dlt + 2 * plane + o) = lo;
    }
  }
  __syncthreads();  // tile consumed before its space holds the sums
  float* red = sh;  // [2][WAVES][E]
  if (sub == 0) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = j + P * i;
      if (e < E) {
        red[w * E + e] = bsum[i];
        red[(WAVES + w) * E + e] = psum[i];
      }
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += WAVES * kWave) {
    float bs = 0.f, ps = 0.f;
    for (int ww = 0; ww < WAVES; ++ww) {
      bs += red[ww * E + e];
      ps += red[(WAVES + ww) * E + e];
    }
    a.bpart[wb * E + e] = bs;
    if (aux) a.ppart[wb * E + e] = ps;
  }
}

// loss = coef * E * sum_e f_e * P_e (a tree sum over experts in a fixed order).
__global__ __launch_bounds__(1024) void aux_loss_kernel(GateBwdArgs a) {
  __shared__ float red[1024];
  const int t = threadIdx.x;
  float term = 0.f;
  if (t < a.E && a.S > 0) {
    const float inv_s = 1.f / static_cast<float>(a.S);
    term = (static_cast<float>(first_count(a, t)) * inv_s) * (a.pe[t] * inv_s);
  }
  red[t] = term;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  if (t == 0) a.aux_loss[0] = a.aux_coef * static_cast<float>(a.E) * red[0];
}

// db and the balance loss side by side (E <= 64), block sb of 1024 threads:
// with dbias, block 0 sums the per-wave-block dL sums into it; the other sums
// the softmax sums into pe and then forms the loss from them (first-choice
// counts), so no block waits for another.
__device__ __forceinline__ void dl_sums_block(const GateBwdArgs& a, int sb, float (*red)[kWave]) {
  if (a.dbias && sb == 0) {
    colsum_cols(a.bpart, a.nb, a.E, a.dbias, 0, red);
    return;
  }
  const float pe = colsum_cols(a.ppart, a.nb, a.E, a.pe, 0, red);
  if (threadIdx.x >= kWave) return;  // the loss is the first wave's (a whole wave)
  const int e = threadIdx.x;
  float term = 0.f;
  if (e < a.E && a.S > 0) {
    const float inv_s = 1.f / static_cast<float>(a.S);
    term = (static_cast<float>(first_count(a, e)) * inv_s) * (pe * inv_s);
  }
  term = wave_sum(term);
  if (e == 0) a.aux_loss[0] = a.aux_coef * static_cast<float>(a.E) * term;
}

// Blocks of the sums above: db if wanted, the loss if wanted.
inline int dl_sums_blocks(const GateBwdArgs& a) {
  return (a.dbias ? 1 : 0) + (a.aux_coef != 0.f && a.aux_loss ? 1 : 0);
}

__global__ __launch_bounds__(1024) void dl_sums_loss_kernel(GateBwdArgs a) {
  __shared__ float red[16][kWave];
  dl_sums_block(a, blockIdx.x, red);
}

// ---------------------------------------------------------------- dW on matrix cores
// gfx950's LDS transpose read (ds_read_b64_tr_b16): within each group of 16
// lanes, lane i receives element i % 4 of the four-element rows addressed by
// lanes i / 4 + 4 j, j = 0..3 (checked on MI355X with an index-filled buffer).
// Two such reads turn a row-major tile of x into the A operand x^T.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ uint2 lds_read_tr16(const uint16_t* p) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p)));
}

// 16-byte piece of row t of a 64 x 64 bf16 tile (128-byte rows, no padding):
// logical piece p sits at p ^ dw_swz(t), so that the 32 rows one transpose read
// touches (4 per lane group, even and odd halves) fall into distinct pieces.
__device__ __forceinline__ int dw_swz(int t) { return ((t >> 1) & 1) | (((t >> 3) & 3) << 1); }

// Block: 256 columns of x (64 per wave) x one token range, walked in 64-token
// chunks that all four waves take together.  Per chunk the block stages the
// chunk's three dL^T planes (E rows of 64 tokens each) in LDS, double
// buffered, and every wave reads its B fragments (B[s][e] = dL^T[e][s]) from
// there; each wave stages its 64 x 64 tile of x as it is (rows of 128 bytes,
// pieces swizzled) and reads the A operand A[j][s] = x[s][j] back through
// transpose reads.  The next chunk's planes and rows are loaded into registers
// right after the chunk's barrier, unconditionally (rows outside the range
// read a valid row and are zeroed on the way to LDS), and stay in flight
// through the products, which wait on LDS only.  4 M tiles (16 columns) x NT N
// tiles (16 experts), K = 32 tokens; each wave stores its own partial sums.
template <int NT>
__global__ __launch_bounds__(kBwdThreads) __attribute__((amdgpu_waves_per_eu(NT <= 4 ? 2 : 1))) void dwg_mfma_kernel(GateBwdArgs a) {
  constexpr int E = 16 * NT;
  constexpr int kRows = 3 * E;                         // plane rows per chunk
  constexpr int kPieces = kRows * 8;                   // 16-byte pieces per chunk
  constexpr int kPer = (kPieces + kBwdThreads - 1) / kBwdThreads;
  __shared__ __align__(16) uint16_t pl[2][kRows * kWave];
  __shared__ __align__(16) uint16_t xt[kBwdWaves][kWave * kWave];
  const int w = threadIdx.x / kWave, lane = lane_id();
  const int g = lane / 16, m = lane % 16;
  const int lr = lane / 8, lp = lane % 8;  // row (of 8) and 16-byte piece this lane loads of x
  // 1-D grid, blocks dealt round-robin to the 8 XCDs (block id mod 8): all
  // column blocks of one token range go to the same XCD and share its L2 copy
  // of that range's dL planes
  const int ncb = (a.d + 4 * kWave - 1) / (4 * kWave);
  const int xcd = blockIdx.x % 8, r8 = blockIdx.x / 8;
  const int split = xcd + 8 * (r8 / ncb);
  if (split >= a.nsplit) return;  // idle block (whole block, before any barrier)
  const int jw = (r8 % ncb) * 4 * kWave + w * kWave;  // this wave's first column
  const bool wcols = jw < a.d;                        // a wave past d stores nothing
  const int jx = wcols ? jw : 0;
  const int64_t sb = static_cast<int64_t>(split) * a.split_tokens;
  const int64_t se = min(static_cast<int64_t>(a.S), sb + a.split_tokens);
  const int nchunks = static_cast<int>((se - sb + kWave - 1) / kWave);
  const uint16_t* x = reinterpret_cast<const uint16_t*>(a.x);
  uint16_t* tile = xt[w];
  const u32x4 zero = {0u, 0u, 0u, 0u};

  f32x4 acc[4][NT];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 rows[8], pv[kPer];
  auto load_next = [&](int c) {
    const int cc = c < nchunks ? c : 0;
    const int64_t s0 = sb + static_cast<int64_t>(cc) * kWave;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int64_t s = s0 + 8 * r + lr;
      rows[r] = *reinterpret_cast<const u32x4*>(x + (s < se ? s : sb) * a.d + jx + 8 * lp);
    }
    // plane rows are contiguous: row q / 8 of the [3 E, s_pad] array, tokens
    // s0 + 8 (q % 8) .. + 8 (zero beyond S)
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q0 = static_cast<int>(threadIdx.x) + i * kBwdThreads;
      const int q = (kPieces % kBwdThreads == 0 || q0 < kPieces) ? q0 : 0;
      pv[i] = *reinterpret_cast<const u32x4*>(a.dlt + static_cast<int64_t>(q / 8) * a.s_pad + s0 + 8 * (q % 8));
    }
  };
  load_next(0);
  for (int c = 0; c < nchunks; ++c) {
    const int64_t s0 = sb + static_cast<int64_t>(c) * kWave;
    uint16_t* pb = pl[c & 1];
    // this chunk's planes and rows into LDS (the planes' buffer was last read
    // two chunks ago, before the previous barrier; the tile's last reads are
    // this wave's own, earlier in its LDS order)
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = static_cast<int>(threadIdx.x) + i * kBwdThreads;
      const int r = q / 8;
      if (kPieces % kBwdThreads == 0 || q < kPieces)
        *reinterpret_cast<u32x4*>(&pb[r * kWave + 8 * ((q % 8) ^ (r & 7))]) = pv[i];
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int t = 8 * r + lr;
      *reinterpret_cast<u32x4*>(&tile[t * kWave + 8 * (lp ^ dw_swz(t))]) = (s0 + t < se) ? rows[r] : zero;
    }
    __syncthreads();
    load_next(c + 1);
    __builtin_amdgcn_sched_barrier(0);
    {  // a wave past d multiplies a valid tile it does not store (no branch around the products)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        u32x4 av[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          // lane q of group g addresses row 32 ks + 8 g + 4 h + q / 4, columns
          // 16 mt + 4 (q % 4) .. + 3; lane m then holds x[32 ks + 8 g + 4 h + j][16 mt + m]
          uint2 half[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int t = 32 * ks + 8 * g + 4 * h + m / 4;
            const int piece = (2 * mt + (m % 4) / 2) ^ dw_swz(t);
            half[h] = lds_read_tr16(&tile[t * kWave + 8 * piece + 4 * (m % 2)]);
          }
          av[mt] = u32x4{half[0].x, half[0].y, half[1].x, half[1].y};
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          u32x4 b3[3];
#pragma unroll
          for (int pn = 0; pn < 3; ++pn) {
            const int r = pn * E + 16 * nt + m;
            b3[pn] = *reinterpret_cast<const u32x4*>(&pb[r * kWave + 8 * ((4 * ks + g) ^ (r & 7))]);
          }
#pragma unroll
          for (int mt = 0; mt < 4; ++mt) {
            acc[mt][nt] = mfma_bf16(av[mt], b3[0], acc[mt][nt]);
            acc[mt][nt] = mfma_bf16(av[mt], b3[1], acc[mt][nt]);
            acc[mt][nt] = mfma_bf16(av[mt], b3[2], acc[mt][nt]);
          }
          __builtin_amdgcn_sched_barrier(0);  // one N tile's fragments live at a time
        }
      }
    }
  }
  // lane (g, m) of tile (mt, nt) holds columns 16 mt + 4 g + i, expert 16 nt + m
  if (wcols) {
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        *reinterpret_cast<f32x4*>(a.wpart + (static_cast<int64_t>(split) * E + 16 * nt + m) * a.d + jw + 16 * mt + 4 * g) =
            acc[mt][nt];
  }
}

// ---------------------------------------------------------------- dx on matrix cores
// Block: 16 tokens per wave (8 or 4 waves) x 256 columns (4 passes of 64);
// blocks are numbered column block first.  dL of the wave's tokens is kept in registers
// in three bf16 parts; the W rows of a pass are staged in LDS, two passes' rows
// in turn (one barrier per pass).  Each lane adds the incoming dx to its two
// 16-byte pieces of the result and stores them.
// Waves per dx block (16 tokens each): up to 64 experts (at most 128
// registers, four waves per SIMD) eight, so that a block's W rows are staged
// in LDS for 128 tokens; more experts take more registers and keep four.
constexpr int dx_waves(int NT) { return NT <= 4 ? 8 : 4; }

template <int NT>
struct DxShape {
  static constexpr int E = 16 * NT;
  static constexpr int KS = (E + 31) / 32;  // K steps of 32 experts (a half step when E % 32 == 16)
  static constexpr int LDW = E + 8;         // padded W row in LDS (bf16)
};

// FULL: all 64 tokens of the block exist (every block but a ragged last one),
// so no token test splits the code: a branch around a load or a store makes
// the compiler wait for every outstanding memory operation (stores and loads
// share one in-order counter).
//
// The product is taken transposed, dx^T = W dL^T: W rows are the A operand and
// the wave's 16 tokens of dL the B operand, so lane (g, m) of a 16 x 16 tile
// ends up with 4 consecutive columns of token m.  A swap of rows between the
// accumulators of tiles 0 and 1 (and of 2 and 3) gives every lane 8
// consecutive columns of its token, and a rotation by 8 lanes within each row
// regroups them so that one store covers 8 tokens x 128 bytes: whole 128-byte
// lines, which is what keeps the store stream fast while the memory is also
// writing back what earlier kernels left dirty.  No LDS transpose.
template <int NT, bool ACC, bool FULL, int DW>
__device__ __forceinline__ void dx_mfma_body(const GateBwdArgs& a, uint16_t* wl) {
  constexpr int E = DxShape<NT>::E, KS = DxShape<NT>::KS, LDW = DxShape<NT>::LDW;
  constexpr int kThreads = DW * kWave;
  const int w = threadIdx.x / kWave, lane = lane_id();
  const int g = lane / 16, m = lane % 16;
  const int ncb = (a.d + 4 * kWave - 1) / (4 * kWave);  // column blocks of 256
  const int64_t tb = blockIdx.x / ncb;                   // block of 16 * DW tokens
  const int64_t s0 = tb * (16 * DW) + 16 * w;           // the wave's first token
  const int64_t sm = s0 + m;                             // this lane's token in the product
  const bool tok_ok = FULL || sm < a.S;
  const uint16_t* wg = reinterpret_cast<const uint16_t*>(a.wg);
  // tokens of this lane's two pieces of dx: 8 h + (m & 7)
  const int64_t sp0 = s0 + (m & 7), sp1 = s0 + 8 + (m & 7);
  const bool ok0 = FULL || sp0 < a.S, ok1 = FULL || sp1 < a.S;
  uint16_t* dxr0 = reinterpret_cast<uint16_t*>(a.dx) + (ok0 ? sp0 : 0) * a.d;
  uint16_t* dxr1 = reinterpret_cast<uint16_t*>(a.dx) + (ok1 ? sp1 : 0) * a.d;
  const u32x4 zero = {0u, 0u, 0u, 0u};

  u32x4 ah[KS], am[KS], al[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int e0 = 32 * ks + 8 * g;
    float vv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (tok_ok && e0 < E) {
      const float4 p0 = *reinterpret_cast<const float4*>(a.dl + sm * E + e0);
      const float4 p1 = *reinterpret_cast<const float4*>(a.dl + sm * E + e0 + 4);
      vv[0] = p0.x; vv[1] = p0.y; vv[2] = p0.z; vv[3] = p0.w;
      vv[4] = p1.x; vv[5] = p1.y; vv[6] = p1.z; vv[7] = p1.w;
    }
    split8(vv, ah[ks], am[ks], al[ks]);
  }
  const int jb = static_cast<int>(blockIdx.x % ncb) * 4 * kWave;
  // Loads are unconditional (clamped addresses; a value past the end is never
  // used), so that no branch hides one from the wait counts, and they are
  // issued a pass ahead: W rows and the incoming dx of pass cb + 1 while pass
  // cb runs.  Vector-memory loads complete in issue order, so the waits for
  // one pass's values leave the next pass's loads in flight.
  constexpr int WPT = (kWave * (E / 8) + kThreads - 1) / kThreads;  // 16-byte pieces per thread
  u32x4 wreg[WPT];
  auto load_w = [&](int j0) {
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int q = min(static_cast<int>(threadIdx.x) + u * kThreads, kWave * (E / 8) - 1);
      const int r = q / (E / 8), p8 = q % (E / 8);
      const int row = min(j0 + r, a.d - 1);
      wreg[u] = *reinterpret_cast<const u32x4*>(wg + static_cast<int64_t>(row) * E + 8 * p8);
    }
  };
  // lane (g, m): piece h of a pass is token 8 h + (m & 7), 8 columns at
  // 32 (m >> 3) + cofs
  const int cofs = 16 * (g & 1) + 8 * (g >> 1), pcol = 32 * (m >> 3) + cofs;
  auto dx_at = [&](int h, int j0) {
    return reinterpret_cast<u32x4*>((h ? dxr1 : dxr0) + min(j0, a.d - kWave) + pcol);
  };
  u32x4 din[2] = {zero, zero}, dnx[2] = {zero, zero};
  if constexpr (ACC) {
#pragma unroll
    for (int p = 0; p < 2; ++p) din[p] = *dx_at(p, jb);
  }
  load_w(jb);
  // unrolled, so that handing the prefetched dx to the next pass is a renaming,
  // not a register move that would wait for the load
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) {
    const int j0 = jb + cb * kWave;
    if (j0 >= a.d) break;  // the same for the whole block
    // W rows double buffered: pass cb - 2 last read this buffer, before the
    // barrier of pass cb - 1, so one barrier per pass suffices
    uint16_t* wb = wl + (cb & 1) * kWave * LDW;
#pragma unroll
    for (int u = 0; u < WPT; ++u) {  // clamped like the loads: a repeated piece rewrites its own value
      const int q = min(static_cast<int>(threadIdx.x) + u * kThreads, kWave * (E / 8) - 1);
      const int r = q / (E / 8), p8 = q % (E / 8);
      *reinterpret_cast<u32x4*>(&wb[r * LDW + 8 * p8]) = wreg[u];
    }
    __syncthreads();
    load_w(j0 + kWave);
    if constexpr (ACC) {
#pragma unroll
      for (int p = 0; p < 2; ++p) dnx[p] = *dx_at(p, j0 + kWave);
    }
    f32x4 acc[4];
    // the W fragments of two tiles read from LDS together, then their products
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      u32x4 bw[2][KS];
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int e0 = 32 * ks + 8 * g;
          bw[q][ks] = e0 < E ? *reinterpret_cast<const u32x4*>(&wb[(16 * (2 * hh + q) + m) * LDW + e0]) : zero;
        }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int nt = 2 * hh + q;
        acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          acc[nt] = mfma_bf16(bw[q][ks], ah[ks], acc[nt]);
          acc[nt] = mfma_bf16(bw[q][ks], am[ks], acc[nt]);
          acc[nt] = mfma_bf16(bw[q][ks], al[ks], acc[nt]);
        }
      }
    }
    // lane (g, m) holds columns 16 nt + 4 g + i of token m.  The permlane16
    // swap exchanges odd rows of its first operand with even rows of its
    // second: lanes of even g keep tile 2p's columns 4 g.. and get tile 2p's
    // 4 (g + 1).. from lane g + 1; lanes of odd g get tile 2p + 1's 4 (g - 1)..
    // and keep their own 4 g.. of it: X (p = 0) and Y (p = 1) hold 8 columns
    // at 32 p + cofs of token m.  (The vector components are copied to scalars
    // first: a bit cast taken straight from a component of an ext-vector reads
    // component 0.)
    float xv[8], yv[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float f0 = acc[0][i], f1 = acc[1][i], f2 = acc[2][i], f3 = acc[3][i];
      const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, f0), __builtin_bit_cast(int, f1),
                                                      false, false);
      const auto q = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, f2), __builtin_bit_cast(int, f3),
                                                      false, false);
      xv[i] = __builtin_bit_cast(float, static_cast<int>(r[0]));
      xv[4 + i] = __builtin_bit_cast(float, static_cast<int>(r[1]));
      yv[i] = __builtin_bit_cast(float, static_cast<int>(q[0]));
      yv[4 + i] = __builtin_bit_cast(float, static_cast<int>(q[1]));
    }
    // piece 0 (tokens 0-7): lanes m < 8 their own X, lanes m >= 8 the Y of lane
    // m - 8; piece 1 (tokens 8-15): lanes m < 8 the X of lane m + 8, lanes
    // m >= 8 their own Y.  Lane m meets lane m +- 8 by a DPP rotation of its
    // 16-lane row by 8.
    const bool lo = m < 8;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float o[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float keep = h == 0 ? xv[i] : yv[i];
        const float moved = __builtin_bit_cast(
            float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, h == 0 ? yv[i] : xv[i]), 0x128, 0xF, 0xF, false));
        o[i] = (h == 0) == lo ? keep : moved;
      }
      if constexpr (ACC) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          o[2 * q] += bf16_lo(din[h][q]);
          o[2 * q + 1] += bf16_hi(din[h][q]);
        }
      }
      if (h == 0 ? ok0 : ok1)
        __builtin_nontemporal_store(u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]),
                                          pack_bf16x2(o[4], o[5]), pack_bf16x2(o[6], o[7])},
                                    dx_at(h, j0));
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) din[p] = dnx[p];
  }
}

// Up to 64 experts the kernel fits four waves per SIMD (at most 128 registers);
// more experts need more registers for the dL planes and take fewer waves.
template <int NT, bool ACC, int DW>
__global__ __launch_bounds__(DW * kWave) __attribute__((amdgpu_waves_per_eu(NT <= 4 ? 4 : 1, NT <= 4 ? 4 : 8)))
void dx_mfma_kernel(GateBwdArgs a) {
  __shared__ __align__(16) uint16_t wl[2 * kWave * DxShape<NT>::LDW];
  const int ncb = (a.d + 4 * kWave - 1) / (4 * kWave);
  if ((static_cast<int64_t>(blockIdx.x / ncb) + 1) * (16 * DW) <= a.S) dx_mfma_body<NT, ACC, true, DW>(a, wl);
  else dx_mfma_body<NT, ACC, false, DW>(a, wl);
}

// ---------------------------------------------------------------- dW, dx on the vector ALUs
// Block (j-tile of 64 columns, token range `split`, expert chunk of EC): x and
// dL tiles of 64 tokens staged in LDS; thread (column jj, expert quarter eg)
// accumulates EC/4 sums, tile by tile.  Partials [split][E][d].
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
  for (int64_t s0 = sb; s0 < se; s0 += kWave) {
    __syncthreads();
    for (int q = t; q < kWave * kWave; q += kBwdThreads) {
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
    for (int tok = 0; tok < kWave; ++tok) {
      const float xv = xs[tok][jj];
#pragma unroll
      for (int i = 0; i < EG; ++i) tacc[i] = fmaf(xv, ds[tok][eg * EG + i], tacc[i]);
    }
#pragma unroll
    for (int i = 0; i < EG; ++i) acc[i] += tacc[i];
  }
  const int jw = j0 + jj;
  if (jw < a.d) {
#pragma unroll
    for (int i = 0; i < EG; ++i) {
      const int e = e0 + eg * EG + i;
      if (e < a.E) a.wpart[(static_cast<int64_t>(split) * a.E + e) * a.d + jw] = acc[i];
    }
  }
}

// dwg[j][e] = sum over the token ranges, in order; blocks past the sums run
// the db / balance-loss sums (sums_in_reduce).
constexpr int kReduceThreads = 1024;

__global__ __launch_bounds__(kReduceThreads) void dwg_reduce_kernel(GateBwdArgs a) {
  const int64_t n = static_cast<int64_t>(a.E) * a.d;
  const int64_t nr = (n + kReduceThreads - 1) / kReduceThreads;
  if (static_cast<int64_t>(blockIdx.x) >= nr) {
    __shared__ float red[16][kWave];
    dl_sums_block(a, static_cast<int>(blockIdx.x - nr), red);
    return;
  }
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kReduceThreads + threadIdx.x;
  if (idx >= n) return;
  const int e = static_cast<int>(idx / a.d), jx = static_cast<int>(idx % a.d);
  // eight ranges' loads in flight at a time; the additions stay in range order
  float v = 0.f;
  int sp = 0;
  for (; sp + 8 <= a.nsplit; sp += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = a.wpart[static_cast<int64_t>(sp + u) * n + idx];
#pragma unroll
    for (int u = 0; u < 8; ++u) v += t[u];
  }
  for (; sp < a.nsplit; ++sp) v += a.wpart[static_cast<int64_t>(sp) * n + idx];
  a.dwg[static_cast<int64_t>(jx) * a.E + e] = v;
}

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
    float wv[EC];
#pragma unroll
    for (int ee = 0; ee < EC; ++ee)
      wv[ee] = (jx < a.d && e0 + ee < a.E) ? load_elem(wg, static_cast<int64_t>(jx) * a.E + e0 + ee) : 0.f;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const float* drow = ds[tg + 4 * i];
#pragma unroll
      for (int ee = 0; ee < EC; ++ee) acc[i] = fmaf(drow[ee], wv[ee], acc[i]);
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
      if (a.accumulate) v += bf16_bits_to_f32(dx[o]);
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
  // up to 16 waves per 64-token block (one pass each) while the sums fit LDS
  constexpr int TP = kWave / P;
  constexpr int WAVES = P <= 32 ? (kWave / TP < 16 ? kWave / TP : 16) : 4;
  const size_t tile = a.dlt ? static_cast<size_t>(kWave) * (a.E + 1) * sizeof(float) : 0;
  const size_t sums = static_cast<size_t>(2 * WAVES) * a.E * sizeof(float);
  const int rows = count_rows(a.S);
  const size_t counts = (a.aux_coef != 0.f && rows <= kCountRowsInline) ? static_cast<size_t>(rows) * a.E * sizeof(int) : 0;
  gate_dl_kernel<P, EPL, WAVES>
      <<<dim3(static_cast<unsigned>(a.nb)), dim3(WAVES * kWave), (tile > sums ? tile : sums) + counts, st>>>(a);
}

static void launch_colsum_f(const float* part, int64_t rows, int E, float* out, hipStream_t st) {
  colsum_kernel<float><<<dim3((E + kWave - 1) / kWave), dim3(1024), 0, st>>>(part, rows, E, out);
}

// The per-block first-choice counts sit right after cnt in the workspace.
hipError_t launch_gate_bwd_dl(const GateBwdArgs& a, hipStream_t st) {
  const bool aux = a.aux_coef != 0.f;
  if (aux) {
    int32_t* cpart = a.cnt + a.E;
    const int64_t cblocks = (static_cast<int64_t>(a.S) + kCountTokens - 1) / kCountTokens;
    if (cblocks > 0)
      aux_counts_kernel<<<dim3(static_cast<unsigned>(cblocks)), dim3(1024), static_cast<size_t>(a.E) * sizeof(int),
                          st>>>(a, cpart);
    if (cblocks > kCountRowsInline)
      colsum_kernel<int32_t><<<dim3((a.E + kWave - 1) / kWave), dim3(1024), 0, st>>>(cpart, cblocks, a.E, a.cnt);
  }
  if (a.nb > 0) {
    const int E = a.E;
    if (E <= 4) launch_dl_t<4, 1>(a, st);
    else if (E <= 8) launch_dl_t<4, 2>(a, st);
    else if (E <= 16) launch_dl_t<4, 4>(a, st);
    else if (E <= 32) launch_dl_t<8, 4>(a, st);
    else if (E <= 64) launch_dl_t<16, 4>(a, st);
    else if (E <= 128) launch_dl_t<32, 4>(a, st);
    else if (E <= 256) launch_dl_t<64, 4>(a, st);
    else if (E <= 512) launch_dl_t<64, 8>(a, st);
    else launch_dl_t<64, 16>(a, st);
  }
  if (a.sums_in_reduce) return hipGetLastError();  // the dW reduction launch takes them
  if (a.E <= kWave && dl_sums_blocks(a) > 0) {
    // db and the loss in one launch
    dl_sums_loss_kernel<<<dim3(dl_sums_blocks(a)), dim3(1024), 0, st>>>(a);
    return hipGetLastError();
  }
  if (a.dbias) launch_colsum_f(a.bpart, a.nb, a.E, a.dbias, st);
  if (aux && a.aux_loss) {
    launch_colsum_f(a.ppart, a.nb, a.E, a.pe, st);
    aux_loss_kernel<<<dim3(1), dim3(1024), 0, st>>>(a);
  }
  return hipGetLastError();
}

constexpr int kDwEC = 64;  // experts per vector-ALU dW block
constexpr int kDxEC = 32;  // experts per register chunk in the vector-ALU dx

template <int NT>
static void launch_dwg_mfma_t(const GateBwdArgs& a, hipStream_t st) {
  const int64_t per_xcd = (a.nsplit + 7) / 8;  // token ranges per XCD
  const dim3 grid(static_cast<unsigned>(8 * per_xcd * ((a.d + 4 * kWave - 1) / (4 * kWave))));
  dwg_mfma_kernel<NT><<<grid, dim3(kBwdThreads), 0, st>>>(a);
}

hipError_t launch_gate_bwd_dwg(const GateBwdArgs& a, hipStream_t st) {
  if (a.nsplit > 0) {
    if (a.mfma_dw) {
      switch (a.E / 16) {
        case 1: launch_dwg_mfma_t<1>(a, st); break;
        case 2: launch_dwg_mfma_t<2>(a, st); break;
        case 3: launch_dwg_mfma_t<3>(a, st); break;
        case 4: launch_dwg_mfma_t<4>(a, st); break;
        case 5: launch_dwg_mfma_t<5>(a, st); break;
        case 6: launch_dwg_mfma_t<6>(a, st); break;
        case 7: launch_dwg_mfma_t<7>(a, st); break;
        default: launch_dwg_mfma_t<8>(a, st); break;
      }
    } else {
      const dim3 grid((a.d + kWave - 1) / kWave, a.nsplit, (a.E + kDwEC - 1) / kDwEC);
      if (a.dtype == 1) dwg_partial_kernel<bf16_t, kDwEC><<<grid, dim3(kBwdThreads), 0, st>>>(a);
      else dwg_partial_kernel<float, kDwEC><<<grid, dim3(kBwdThreads), 0, st>>>(a);
    }
  }
  const int64_t n = static_cast<int64_t>(a.E) * a.d;
  const int64_t nr = (n + kReduceThreads - 1) / kReduceThreads;
  const int64_t extra = a.sums_in_reduce ? dl_sums_blocks(a) : 0;
  dwg_reduce_kernel<<<dim3(static_cast<unsigned>(nr + extra)), dim3(kReduceThreads), 0, st>>>(a);
  return hipGetLastError();
}

template <int NT>
static void launch_dx_mfma_t(const GateBwdArgs& a, hipStream_t st) {
  // 1-D grid, the column blocks of one 64-token block consecutive, so that
  // they run side by side and whole rows of dx stream together
  constexpr int DW = dx_waves(NT);
  const int64_t tblocks = (static_cast<int64_t>(a.S) + 16 * DW - 1) / (16 * DW);
  const dim3 grid(static_cast<unsigned>(static_cast<int64_t>((a.d + 4 * kWave - 1) / (4 * kWave)) * tblocks));
  if (a.accumulate) dx_mfma_kernel<NT, true, DW><<<grid, dim3(DW * kWave), 0, st>>>(a);
  else dx_mfma_kernel<NT, false, DW><<<grid, dim3(DW * kWave), 0, st>>>(a);
}

hipError_t launch_gate_bwd_dx(const GateBwdArgs& a, hipStream_t st) {
  if (a.nb == 0) return hipSuccess;
  if (a.mfma_dx) {
    switch (a.E / 16) {
      case 1: launch_dx_mfma_t<1>(a, st); break;
      case 2: launch_dx_mfma_t<2>(a, st); break;
      case 3: launch_dx_mfma_t<3>(a, st); break;
      case 4: launch_dx_mfma_t<4>(a, st); break;
      case 5: launch_dx_mfma_t<5>(a, st); break;
      case 6: launch_dx_mfma_t<6>(a, st); break;
      case 7: launch_dx_mfma_t<7>(a, st); break;
      default: launch_dx_mfma_t<8>(a, st); break;
    }
    return hipGetLastError();
  }
  const dim3 grid((a.d + kWave - 1) / kWave, a.nb);
  if (a.dtype == 1) dx_kernel<bf16_t, kDxEC><<<grid, dim3(kBwdThreads), 0, st>>>(a);
  else dx_kernel<float, kDxEC><<<grid, dim3(kBwdThreads), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace hetumoe
