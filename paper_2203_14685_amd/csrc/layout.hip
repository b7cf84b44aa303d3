// Layout-transform kernels for gfx950: steps 2 and 6 of Algorithm 1 and their
// gradients.  Every output row has exactly one writer, so there are no atomics
// and results are bitwise reproducible.  Outputs indexed by token (combine,
// dispatch backward) are gathers; outputs indexed by expert slot (dispatch,
// combine backward) are gathers over slots for k = 1 and token-major scatters
// for k > 1, so that each token row is read once.
//
// Two row forms.  The flat form (the [E,C,d] gathers for k = 1, and the
// token-order gathers for k <= 2 over rows of up to 2 KiB) gives every thread
// one 16-byte chunk of the flattened output per step, two steps per thread, so
// a block of 512 threads writes 16 KiB and lives briefly.  The wave form gives
// one wavefront one output row, walked in 16-byte chunks (64 lanes x 16 B =
// 1 KiB per instruction) with up to kUnroll loads per lane in flight before
// the first store.  On MI355X many short-lived waves with few stores each kept
// more writes in flight than long row walks (a 1 GiB fill: 6.8 TB/s with one
// store per thread against 5.7 TB/s with eight), which is why the writers of
// [E,C,d] use the flat form; the wave form stays where it measured faster
// (token rows longer than 2 KiB, k >= 3, and the token-major scatters).
// Every output row is written with non-temporal stores: the buffers are far
// larger than the 256 MB Infinity Cache, and plain stores leave dirty lines there
// whose write-back then slows whichever kernel runs next (measured: dispatch
// after a plain-store producer ~25% slower than after a streaming one).  The
// wave, short-row and token-major forms also read their source rows with
// non-temporal loads (each row is read once; 2-7 % faster), the flat forms with
// plain loads (1-2 % faster there).
#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

constexpr int kUnroll = 8;
// Waves per block, one row per wave.  Large blocks measured faster on MI355X for
// these gathers (16 waves for the [E,C,d] writers); the combine kernels keep 4
// so that their fp32 accumulators fit the register budget without spilling.
constexpr int kWideWaves = 16;
constexpr int kCombineWaves = 4;
// The token-major combine backward with dw holds ~126 VGPRs, four waves per
// SIMD: 16-wave blocks would run one at a time per CU.  Blocks of 8 balance
// small batches better (workload of 8192 tokens, k = 2: 20.5 -> 18.5 us).
constexpr int kBwdScatterWaves = 8;

__device__ __forceinline__ void store_nt(u32x4* p, const u32x4& v) { __builtin_nontemporal_store(v, p); }

// ---------------------------------------------------------------- flat form
constexpr int kFlatThreads = 512;
constexpr int kFlatPer = 2;                          // chunks per thread
constexpr int kFlatChunks = kFlatThreads * kFlatPer;  // chunks per block
constexpr int kFlatWaves = kFlatThreads / kWave;

// Row and column of chunk gb + off of a flattened [rows, nch] output, where gb
// is the block's first chunk (row_b, col_b precomputed) and off < kFlatChunks.
// POW2: nch = 1 << lg.
template <bool POW2>
__device__ __forceinline__ void flat_pos(int64_t gb, int64_t row_b, int col_b, int off, int nch, int lg, int64_t& row,
                                         int& col) {
  if constexpr (POW2) {
    const int64_t g = gb + off;
    row = g >> lg;
    col = static_cast<int>(g & (nch - 1));
  } else {
    const unsigned t = static_cast<unsigned>(col_b + off);
    const unsigned q = t / static_cast<unsigned>(nch);
    row = row_b + q;
    col = static_cast<int>(t - q * static_cast<unsigned>(nch));
  }
}

// ---------------------------------------------------------------- dispatch
// xe[row] = x[slot_src[row] / k], or zeros for an empty slot.  Flat form for
// k = 1 (k > 1 uses the token-major scatter further down).
template <bool POW2>
__global__ __launch_bounds__(kFlatThreads) void dispatch_flat_kernel(RowArgs a, int lg, int64_t total) {
  const int nch = a.nch;
  const int64_t gb = static_cast<int64_t>(blockIdx.x) * kFlatChunks;
  const int64_t row_b = POW2 ? 0 : gb / nch;
  const int col_b = POW2 ? 0 : static_cast<int>(gb - row_b * nch);
  const u32x4* x = reinterpret_cast<const u32x4*>(a.src);
  u32x4* xe = reinterpret_cast<u32x4*>(a.dst);
  u32x4 v[kFlatPer];
#pragma unroll
  for (int u = 0; u < kFlatPer; ++u) {
    const int off = u * kFlatThreads + static_cast<int>(threadIdx.x);
    int64_t row;
    int col;
    flat_pos<POW2>(gb, row_b, col_b, off, nch, lg, row, col);
    // entries outside [0, S) are out of contract and treated as empty slots
    const int src = gb + off < total ? a.slot_src[row] : -1;
    v[u] = u32x4{0u, 0u, 0u, 0u};
    if (src >= 0 && src < a.S) v[u] = x[static_cast<int64_t>(src) * nch + col];
  }
#pragma unroll
  for (int u = 0; u < kFlatPer; ++u) {
    const int64_t g = gb + u * kFlatThreads + static_cast<int>(threadIdx.x);
    if (g < total) store_nt(xe + g, v[u]);
  }
}

// ---------------------------------------------------------------- combine
// y[s] = sum_{r kept} w[s,r] * ye[ids[s,r], slots[s,r]]  (WEIGHTED)
// dx[s] = sum_{r kept} dxe[ids[s,r], slots[s,r]]        (!WEIGHTED)
// fp32 accumulation in r order, one rounding to T.
template <typename T, bool WEIGHTED>
__global__ __launch_bounds__(kCombineWaves * kWave) void combine_kernel(RowArgs a) {
  constexpr int kEl = Chunk<T>::kElems;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kCombineWaves + threadIdx.x / kWave;
  if (s >= a.rows) return;
  const int lane = lane_id();
  const int nch = a.nch, k = a.k;
  const u32x4* ye = reinterpret_cast<const u32x4*>(a.src);
  u32x4* out = reinterpret_cast<u32x4*>(a.dst) + s * nch;
  for (int base = 0; base < nch; base += kWave * kUnroll) {
    float acc[kUnroll][kEl];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int q = 0; q < kEl; ++q) acc[u][q] = 0.f;
    for (int r = 0; r < k; ++r) {
      const int slot = a.slots[s * k + r];
      const int e = a.ids[s * k + r];
      // dropped choices (slot -1) and out-of-contract entries contribute nothing
      if (slot < 0 || slot >= a.C || e < 0 || e >= a.E) continue;
      const float w = WEIGHTED ? a.weights[s * k + r] : 1.f;
      const u32x4* srow = ye + (static_cast<int64_t>(e) * a.C + slot) * nch;
      u32x4 v[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int i = base + u * kWave + lane;
        // each source row is read once: streaming loads, as in the short and
        // token-major forms (the flat forms measured slower with them)
        if (i < nch) v[u] = __builtin_nontemporal_load(&srow[i]);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int i = base + u * kWave + lane;
        if (i < nch) {
          float f[kEl];
          Chunk<T>::unpack(v[u], f);
#pragma unroll
          for (int q = 0; q < kEl; ++q) acc[u][q] = WEIGHTED ? fmaf(w, f[q], acc[u][q]) : acc[u][q] + f[q];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = base + u * kWave + lane;
      if (i < nch) store_nt(out + i, Chunk<T>::pack(acc[u]));
    }
  }
}

// Short rows (CPR x 64 chunks per row, CPR in {1, 2, 4}): one wave takes
// RPW = 8 / CPR tokens so that every lane still has 8 loads in flight.  All of
// a rank's slot, id and weight reads come first; the row loads are then issued
// unconditionally (a dropped choice reads row 0 of the expert buffer, which
// needs E * C > 0, and its value is discarded), so no load waits behind a
// branch on another load's result.
template <typename T, bool WEIGHTED, int CPR>
__global__ __launch_bounds__(kCombineWaves * kWave) void combine_short_kernel(RowArgs a) {
  constexpr int kEl = Chunk<T>::kElems;
  constexpr int RPW = 8 / CPR;
  constexpr int nch = CPR * kWave;
  const int64_t s0 = (static_cast<int64_t>(blockIdx.x) * kCombineWaves + threadIdx.x / kWave) * RPW;
  if (s0 >= a.rows) return;
  const int lane = lane_id();
  const int k = a.k;
  const u32x4* ye = reinterpret_cast<const u32x4*>(a.src);
  u32x4* out = reinterpret_cast<u32x4*>(a.dst);
  float acc[8][kEl];
#pragma unroll
  for (int u = 0; u < 8; ++u)
#pragma unroll
    for (int q = 0; q < kEl; ++q) acc[u][q] = 0.f;
  for (int r = 0; r < k; ++r) {
    int64_t rowoff[RPW];
    float w[RPW];
    bool ok[RPW];
#pragma unroll
    for (int t = 0; t < RPW; ++t) {
      const int64_t s = min(s0 + t, a.rows - 1);
      const int slot = a.slots[s * k + r];
      const int e = a.ids[s * k + r];
      w[t] = WEIGHTED ? a.weights[s * k + r] : 1.f;
      ok[t] = (s0 + t < a.rows) && slot >= 0 && slot < a.C && e >= 0 && e < a.E;
      rowoff[t] = ok[t] ? (static_cast<int64_t>(e) * a.C + slot) * nch : 0;
    }
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(&ye[rowoff[u / CPR] + (u % CPR) * kWave + lane]);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (ok[u / CPR]) {
        float f[kEl];
        Chunk<T>::unpack(v[u], f);
#pragma unroll
        for (int q = 0; q < kEl; ++q)
          acc[u][q] = WEIGHTED ? fmaf(w[u / CPR], f[q], acc[u][q]) : acc[u][q] + f[q];
      }
    }
  }
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int64_t s = s0 + u / CPR;
    if (s < a.rows) store_nt(out + s * nch + (u % CPR) * kWave + lane, Chunk<T>::pack(acc[u]));
  }
}

// Flat form of the two above for k <= KMAX <= 2: each thread combines one
// 16-byte chunk of a token row per step.  Every load of both steps is issued
// before the first store: vector loads and stores retire in order on one
// counter, so a store between two loads makes the second wait for it
// (measured at 2 KiB rows, k = 2: 14.1 -> 13.3 us).  At 4 and 8 KiB rows
// with k = 1 this form, run alone, beat the wave forms (31.0 against 39.4 us,
// 157 against 160 us), but was slower in the pass, right after the dispatch's
// streaming stores (51.7 against 43.6 us, 176.9 against 164.6 us).
template <typename T, bool POW2, bool WEIGHTED, int KMAX>
__global__ __launch_bounds__(kFlatThreads) void combine_flat_kernel(RowArgs a, int lg, int64_t total) {
  constexpr int kEl = Chunk<T>::kElems;
  const int nch = a.nch, k = a.k;
  const int64_t gb = static_cast<int64_t>(blockIdx.x) * kFlatChunks;
  const int64_t row_b = POW2 ? 0 : gb / nch;
  const int col_b = POW2 ? 0 : static_cast<int>(gb - row_b * nch);
  const u32x4* ye = reinterpret_cast<const u32x4*>(a.src);
  u32x4* out = reinterpret_cast<u32x4*>(a.dst);
  u32x4 v[kFlatPer][KMAX];
  float w[kFlatPer][KMAX];
  bool ok[kFlatPer][KMAX];
#pragma unroll
  for (int u = 0; u < kFlatPer; ++u) {
    const int off = u * kFlatThreads + static_cast<int>(threadIdx.x);
    const bool in = gb + off < total;
    int64_t s;
    int col;
    flat_pos<POW2>(gb, row_b, col_b, off, nch, lg, s, col);
#pragma unroll
    for (int r = 0; r < KMAX; ++r) {
      ok[u][r] = false;
      w[u][r] = 1.f;
      v[u][r] = u32x4{0u, 0u, 0u, 0u};
      if (in && r < k) {
        const int slot = a.slots[s * k + r];
        const int e = a.ids[s * k + r];
        // dropped choices (slot -1) and out-of-contract entries contribute nothing
        ok[u][r] = slot >= 0 && slot < a.C && e >= 0 && e < a.E;
        if (WEIGHTED) w[u][r] = a.weights[s * k + r];
        if (ok[u][r]) v[u][r] = ye[(static_cast<int64_t>(e) * a.C + slot) * nch + col];
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kFlatPer; ++u) {
    const int off = u * kFlatThreads + static_cast<int>(threadIdx.x);
    if (gb + off >= total) continue;
    float acc[kEl];
#pragma unroll
    for (int q = 0; q < kEl; ++q) acc[q] = 0.f;
#pragma unroll
    for (int r = 0; r < KMAX; ++r) {
      if (!ok[u][r]) continue;
      float f[kEl];
      Chunk<T>::unpack(v[u][r], f);
#pragma unroll
      for (int q = 0; q < kEl; ++q) acc[q] = WEIGHTED ? fmaf(w[u][r], f[q], acc[q]) : acc[q] + f[q];
    }
    store_nt(out + gb + off, Chunk<T>::pack(acc));
  }
}

// ---------------------------------------------------------------- combine backward
// Rows [0, rows): dye[row] = w[src] * dy[src / k] (zeros for an empty slot) and,
// with DW, dw[src] = <dy[src / k], ye[row]>.  Blocks past the row blocks clear
// dw of dropped choices.
template <typename T, bool DW>
__global__ __launch_bounds__(kWideWaves * kWave) void combine_bwd_kernel(RowArgs a, int64_t row_blocks) {
  constexpr int kEl = Chunk<T>::kElems;
  if (static_cast<int64_t>(blockIdx.x) >= row_blocks) {
    if constexpr (DW) {
      const int64_t i = (static_cast<int64_t>(blockIdx.x) - row_blocks) * (kWideWaves * kWave) + threadIdx.x;
      if (i < static_cast<int64_t>(a.S) * a.k && a.slots[i] < 0) a.dw[i] = 0.f;
    }
    return;
  }
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kWideWaves + threadIdx.x / kWave;
  if (row >= a.rows) return;
  const int lane = lane_id();
  const int nch = a.nch;
  const int src = a.slot_src[row];
  u32x4* dst = reinterpret_cast<u32x4*>(a.dst) + row * nch;
  if (src < 0 || src >= a.S * a.k) {  // empty (or out-of-contract) slot
    const u32x4 z = {0u, 0u, 0u, 0u};
    for (int i = lane; i < nch; i += kWave) store_nt(dst + i, z);
    return;
  }
  const float w = a.weights[src];
  const u32x4* dyrow = reinterpret_cast<const u32x4*>(a.src) + static_cast<int64_t>(src / a.k) * nch;
  const u32x4* yerow = reinterpret_cast<const u32x4*>(a.aux) + row * nch;
  float dot = 0.f;
  for (int base = 0; base < nch; base += kWave * kUnroll) {
    u32x4 v[kUnroll];
    u32x4 ve[DW ? kUnroll : 1];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = base + u * kWave + lane;
      if (i < nch) {
        v[u] = dyrow[i];
        if constexpr (DW) ve[u] = yerow[i];
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = base + u * kWave + lane;
      if (i < nch) {
        float f[kEl];
        Chunk<T>::unpack(v[u], f);
        if constexpr (DW) {
          float g[kEl];
          Chunk<T>::unpack(ve[u], g);
#pragma unroll
          for (int q = 0; q < kEl; ++q) dot = fmaf(f[q], g[q], dot);
        }
#pragma unroll
        for (int q = 0; q < kEl; ++q) f[q] *= w;
        store_nt(dst + i, Chunk<T>::pack(f));
      }
    }
  }
  if constexpr (DW) {
    dot = wave_sum(dot);
    if (lane == 0) a.dw[src] = dot;
  }
}

// Flat form of the kernel above for k = 1.  With DW the row length must be a
// power of two between 64 chunks (one wave) and kFlatChunks, so that every
// wave lies inside one row and every row inside one block: each wave sums its
// part of <dy, ye>, and one thread per row adds the parts of its waves in
// order.  Blocks past the row blocks clear dw of dropped choices.
template <typename T, bool POW2, bool DW>
__global__ __launch_bounds__(kFlatThreads) void combine_bwd_flat_kernel(RowArgs a, int lg, int64_t total,
                                                                        int64_t row_blocks) {
  constexpr int kEl = Chunk<T>::kElems;
  if (static_cast<int64_t>(blockIdx.x) >= row_blocks) {
    if constexpr (DW) {
      const int64_t i = (static_cast<int64_t>(blockIdx.x) - row_blocks) * kFlatThreads + threadIdx.x;
      if (i < a.S && a.slots[i] < 0) a.dw[i] = 0.f;
    }
    return;
  }
  const int nch = a.nch;
  const int64_t gb = static_cast<int64_t>(blockIdx.x) * kFlatChunks;
  const int64_t row_b = POW2 ? 0 : gb / nch;
  const int col_b = POW2 ? 0 : static_cast<int>(gb - row_b * nch);
  const u32x4* dy = reinterpret_cast<const u32x4*>(a.src);
  const u32x4* ye = reinterpret_cast<const u32x4*>(a.aux);
  u32x4* dye = reinterpret_cast<u32x4*>(a.dst);
  u32x4 v[kFlatPer];
  u32x4 ve[DW ? kFlatPer : 1];
  float w[kFlatPer];
  bool ok[kFlatPer];
#pragma unroll
  for (int u = 0; u < kFlatPer; ++u) {
    const int off = u * kFlatThreads + static_cast<int>(threadIdx.x);
    int64_t row;
    int col;
    flat_pos<POW2>(gb, row_b, col_b, off, nch, lg, row, col);
    // entries outside [0, S) are out of contract and treated as empty slots
    const int src = gb + off < total ? a.slot_src[row] : -1;
    ok[u] = src >= 0 && src < a.S;
    v[u] = u32x4{0u, 0u, 0u, 0u};
    w[u] = 0.f;
    if constexpr (DW) ve[u] = u32x4{0u, 0u, 0u, 0u};
    if (ok[u]) {
      v[u] = dy[static_cast<int64_t>(src) * nch + col];
      w[u] = a.weights[src];
      if constexpr (DW) ve[u] = ye[gb + off];
    }
  }
  float dot[kFlatPer];
#pragma unroll
  for (int u = 0; u < kFlatPer; ++u) {
    const int64_t g = gb + u * kFlatThreads + static_cast<int>(threadIdx.x);
    dot[u] = 0.f;
    if (g >= total) continue;
    if (!ok[u]) {  // empty slot: zeros, no arithmetic
      store_nt(dye + g, u32x4{0u, 0u, 0u, 0u});
      continue;
    }
    float f[kEl];
    Chunk<T>::unpack(v[u], f);
    if constexpr (DW) {
      float gq[kEl];
      Chunk<T>::unpack(ve[u], gq);
#pragma unroll
      for (int q = 0; q < kEl; ++q) dot[u] = fmaf(f[q], gq[q], dot[u]);
    }
#pragma unroll
    for (int q = 0; q < kEl; ++q) f[q] *= w[u];
    store_nt(dye + g, Chunk<T>::pack(f));
  }
  if constexpr (DW) {
    __shared__ float part[kFlatPer * kFlatWaves];  // [u][wave]: chunk offset / 64
    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int u = 0; u < kFlatPer; ++u) {
      const float t = wave_sum(dot[u]);
      if (lane_id() == 0) part[u * kFlatWaves + wave] = t;
    }
    __syncthreads();
    const int rows_here = kFlatChunks >> lg;
    const int parts = nch / kWave;
    if (static_cast<int>(threadIdx.x) < rows_here) {
      const int64_t row = (gb >> lg) + threadIdx.x;
      if (row < a.rows) {
        float t = 0.f;
        for (int j = 0; j < parts; ++j) t += part[threadIdx.x * parts + j];
        const int src = a.slot_src[row];
        if (src >= 0 && src < a.S) a.dw[src] = t;
      }
    }
  }
}

// ---------------------------------------------------------------- token-major forms (k > 1)
// With several choices per token, the slot-major gathers above read each token
// row once per kept choice.  These forms read it once: blocks [0, tok_blocks)
// take one token per wave and write (or, backward, scale and dot) its kept
// rows; the remaining blocks stride over the expert slots and zero the empty
// ones.  Each output row still has exactly one writer.
constexpr int kZeroBlocks = 1024;

__device__ __forceinline__ void zero_empty_rows(const RowArgs& a, int64_t first_wave, int64_t nwaves, int lane) {
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (int64_t row = first_wave; row < a.rows; row += nwaves) {
    const int src = a.slot_src[row];
    if (src >= 0 && src < a.S * a.k) continue;
    u32x4* dst = reinterpret_cast<u32x4*>(a.dst) + row * a.nch;
    for (int i = lane; i < a.nch; i += kWave) store_nt(dst + i, z);
  }
}

// xe[ids[s,r], slots[s,r]] = x[s] for every kept (s, r); empty slots zero.
__global__ __launch_bounds__(kWideWaves * kWave) void dispatch_scatter_kernel(RowArgs a, int64_t tok_blocks) {
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  if (static_cast<int64_t>(blockIdx.x) >= tok_blocks) {
    zero_empty_rows(a, (static_cast<int64_t>(blockIdx.x) - tok_blocks) * kWideWaves + wave,
                    static_cast<int64_t>(gridDim.x - tok_blocks) * kWideWaves, lane);
    return;
  }
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kWideWaves + wave;
  if (s >= a.S) return;
  const int nch = a.nch, k = a.k;
  const u32x4* srow = reinterpret_cast<const u32x4*>(a.src) + s * nch;
  for (int base = 0; base < nch; base += kWave * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = base + u * kWave + lane;
      if (i < nch) v[u] = __builtin_nontemporal_load(&srow[i]);
    }
    for (int r = 0; r < k; ++r) {
      const int slot = a.slots[s * k + r];
      const int e = a.ids[s * k + r];
      if (slot < 0 || slot >= a.C || e < 0 || e >= a.E) continue;
      u32x4* dst = reinterpret_cast<u32x4*>(a.dst) + (static_cast<int64_t>(e) * a.C + slot) * nch;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int i = base + u * kWave + lane;
        if (i < nch) store_nt(dst + i, v[u]);
      }
    }
  }
}

// For every kept (s, r): dye[ids, slots] = w[s,r] * dy[s] and, with DW,
// dw[s,r] = <dy[s], ye[ids, slots]>; dropped choices get dw = 0; empty slots
// of dye are zero.  One wave per token walks the row in steps of 4 chunks per
// lane and issues the loads of up to 4 choices' ye rows together.
template <typename T, bool DW>
__global__ __launch_bounds__(kBwdScatterWaves * kWave) void combine_bwd_scatter_kernel(RowArgs a, int64_t tok_blocks) {
  constexpr int kEl = Chunk<T>::kElems;
  constexpr int kU = 4;   // chunks per lane per step
  constexpr int kRG = 4;  // choices whose rows are loaded together
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  if (static_cast<int64_t>(blockIdx.x) >= tok_blocks) {
    zero_empty_rows(a, (static_cast<int64_t>(blockIdx.x) - tok_blocks) * kBwdScatterWaves + wave,
                    static_cast<int64_t>(gridDim.x - tok_blocks) * kBwdScatterWaves, lane);
    return;
  }
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kBwdScatterWaves + wave;
  if (s >= a.S) return;
  const int nch = a.nch, k = a.k;
  const u32x4* dyrow = reinterpret_cast<const u32x4*>(a.src) + s * nch;
  float dot[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) dot[r] = 0.f;
  for (int base = 0; base < nch; base += kWave * kU) {
    u32x4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int i = base + u * kWave + lane;
      if (i < nch) v[u] = __builtin_nontemporal_load(&dyrow[i]);
    }
#pragma unroll
    for (int r0 = 0; r0 < 8; r0 += kRG) {
      if (r0 >= k) break;
      int64_t row[kRG];
      bool kept[kRG];
      u32x4 ve[DW ? kRG : 1][kU];
#pragma unroll
      for (int j = 0; j < kRG; ++j) {
        const int r = r0 + j;
        const int slot = (r < k) ? a.slots[s * k + r] : -1;
        const int e = (r < k) ? a.ids[s * k + r] : -1;
        kept[j] = slot >= 0 && slot < a.C && e >= 0 && e < a.E;
        row[j] = kept[j] ? static_cast<int64_t>(e) * a.C + slot : 0;
        if constexpr (DW) {
          const u32x4* yerow = reinterpret_cast<const u32x4*>(a.aux) + row[j] * nch;
#pragma unroll
          for (int u = 0; u < kU; ++u) {
            const int i = base + u * kWave + lane;
            if (kept[j] && i < nch) ve[j][u] = __builtin_nontemporal_load(&yerow[i]);
          }
        }
      }
#pragma unroll
      for (int j = 0; j < kRG; ++j) {
        if (!kept[j]) continue;
        const float w = a.weights[s * k + r0 + j];
        u32x4* dst = reinterpret_cast<u32x4*>(a.dst) + row[j] * nch;
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const int i = base + u * kWave + lane;
          if (i < nch) {
            float f[kEl];
            Chunk<T>::unpack(v[u], f);
            if constexpr (DW) {
              float gq[kEl];
              Chunk<T>::unpack(ve[j][u], gq);
#pragma unroll
              for (int q = 0; q < kEl; ++q) dot[r0 + j] = fmaf(f[q], gq[q], dot[r0 + j]);
            }
#pragma unroll
            for (int q = 0; q < kEl; ++q) f[q] *= w;
            store_nt(dst + i, Chunk<T>::pack(f));
          }
        }
      }
    }
  }
  if constexpr (DW) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      if (r >= k) break;
      const float t = wave_sum(dot[r]);
      if (lane == 0) a.dw[s * k + r] = (a.slots[s * k + r] >= 0) ? t : 0.f;
    }
  }
}

// ---------------------------------------------------------------- launchers
static inline unsigned blocks_for_rows(int64_t rows, int waves) {
  return static_cast<unsigned>((rows + waves - 1) / waves);
}

static unsigned zero_blocks(int64_t rows, int waves = kWideWaves) {
  const int64_t b = (rows + waves - 1) / waves;
  const int64_t cap = static_cast<int64_t>(kZeroBlocks) * kWideWaves / waves;
  return static_cast<unsigned>(b < cap ? b : cap);
}

// log2(n) for a power of two, else -1
static inline int pow2_log(int n) {
  if (n <= 0 || (n & (n - 1)) != 0) return -1;
  int lg = 0;
  while ((1 << lg) < n) ++lg;
  return lg;
}

static inline unsigned flat_blocks(int64_t total) {
  return static_cast<unsigned>((total + kFlatChunks - 1) / kFlatChunks);
}

hipError_t launch_dispatch(const RowArgs& a, hipStream_t st) {
  if (a.k > 1) {
    const int64_t tok_blocks = (static_cast<int64_t>(a.S) + kWideWaves - 1) / kWideWaves;
    const unsigned grid = static_cast<unsigned>(tok_blocks) + zero_blocks(a.rows);
    if (grid == 0) return hipSuccess;
    dispatch_scatter_kernel<<<dim3(grid), dim3(kWideWaves * kWave), 0, st>>>(a, tok_blocks);
    return hipGetLastError();
  }
  const int64_t total = a.rows * a.nch;
  if (total == 0) return hipSuccess;
  const int lg = pow2_log(a.nch);
  const dim3 grid(flat_blocks(total)), block(kFlatThreads);
  if (lg >= 0) dispatch_flat_kernel<true><<<grid, block, 0, st>>>(a, lg, total);
  else dispatch_flat_kernel<false><<<grid, block, 0, st>>>(a, lg, total);
  return hipGetLastError();
}

template <typename T, bool WEIGHTED>
static void launch_combine_short(const RowArgs& a, hipStream_t st) {
  const int cpr = a.nch / kWave, rpw = 8 / cpr;
  const dim3 grid(blocks_for_rows((a.rows + rpw - 1) / rpw, kCombineWaves)), block(kCombineWaves * kWave);
  if (cpr == 1) combine_short_kernel<T, WEIGHTED, 1><<<grid, block, 0, st>>>(a);
  else if (cpr == 2) combine_short_kernel<T, WEIGHTED, 2><<<grid, block, 0, st>>>(a);
  else combine_short_kernel<T, WEIGHTED, 4><<<grid, block, 0, st>>>(a);
}

template <typename T, bool POW2, bool WEIGHTED>
static void launch_combine_flat_t(const RowArgs& a, int lg, int64_t total, hipStream_t st) {
  const dim3 grid(flat_blocks(total)), block(kFlatThreads);
  if (a.k == 1) combine_flat_kernel<T, POW2, WEIGHTED, 1><<<grid, block, 0, st>>>(a, lg, total);
  else combine_flat_kernel<T, POW2, WEIGHTED, 2><<<grid, block, 0, st>>>(a, lg, total);
}

template <typename T>
static void launch_combine_flat(const RowArgs& a, bool weighted, hipStream_t st) {
  const int64_t total = a.rows * a.nch;
  const int lg = pow2_log(a.nch);
  if (lg >= 0) {
    if (weighted) launch_combine_flat_t<T, true, true>(a, lg, total, st);
    else launch_combine_flat_t<T, true, false>(a, lg, total, st);
  } else {
    if (weighted) launch_combine_flat_t<T, false, true>(a, lg, total, st);
    else launch_combine_flat_t<T, false, false>(a, lg, total, st);
  }
}

hipError_t launch_combine(const RowArgs& a, bool weighted, hipStream_t st) {
  if (a.rows == 0 || a.nch == 0) return hipSuccess;
  // k <= 2 over rows of up to 2 KiB: flat form (measured 7-15 % faster than
  // the wave forms at 1 and 2 KiB rows; slower in the pass at 4 and 8 KiB rows,
  // and slower at k = 4)
  if (a.k <= 2 && a.nch <= 128) {
    if (a.dtype == 1) launch_combine_flat<bf16_t>(a, weighted, st);
    else launch_combine_flat<float>(a, weighted, st);
    return hipGetLastError();
  }
  // short rows: several tokens per wave (measured 9-11 % faster at 2 and 4 KiB
  // rows); longer rows: one token per wave
  if ((a.nch == 64 || a.nch == 128 || a.nch == 256) && static_cast<int64_t>(a.E) * a.C > 0) {
    if (a.dtype == 1) {
      if (weighted) launch_combine_short<bf16_t, true>(a, st);
      else launch_combine_short<bf16_t, false>(a, st);
    } else {
      if (weighted) launch_combine_short<float, true>(a, st);
      else launch_combine_short<float, false>(a, st);
    }
    return hipGetLastError();
  }
  const dim3 grid(blocks_for_rows(a.rows, kCombineWaves)), block(kCombineWaves * kWave);
  if (a.dtype == 1) {
    if (weighted) combine_kernel<bf16_t, true><<<grid, block, 0, st>>>(a);
    else combine_kernel<bf16_t, false><<<grid, block, 0, st>>>(a);
  } else {
    if (weighted) combine_kernel<float, true><<<grid, block, 0, st>>>(a);
    else combine_kernel<float, false><<<grid, block, 0, st>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_combine_bwd(const RowArgs& a, hipStream_t st) {
  constexpr int kThreads = kWideWaves * kWave;
  if (a.k > 1) {
    const int64_t tok_blocks = (static_cast<int64_t>(a.S) + kBwdScatterWaves - 1) / kBwdScatterWaves;
    const unsigned grid = static_cast<unsigned>(tok_blocks) + zero_blocks(a.rows, kBwdScatterWaves);
    if (grid == 0) return hipSuccess;
    const dim3 block(kBwdScatterWaves * kWave);
    if (a.dtype == 1) {
      if (a.dw) combine_bwd_scatter_kernel<bf16_t, true><<<dim3(grid), block, 0, st>>>(a, tok_blocks);
      else combine_bwd_scatter_kernel<bf16_t, false><<<dim3(grid), block, 0, st>>>(a, tok_blocks);
    } else {
      if (a.dw) combine_bwd_scatter_kernel<float, true><<<dim3(grid), block, 0, st>>>(a, tok_blocks);
      else combine_bwd_scatter_kernel<float, false><<<dim3(grid), block, 0, st>>>(a, tok_blocks);
    }
    return hipGetLastError();
  }
  // k = 1: flat form, with dw where a row is a power of two of 64 to
  // kFlatChunks chunks (else the wave form below)
  const int lg = pow2_log(a.nch);
  if (!a.dw || (lg >= 6 && a.nch <= kFlatChunks)) {
    const int64_t total = a.rows * a.nch;
    const int64_t row_blocks = flat_blocks(total);
    const int64_t dw_blocks = a.dw ? (static_cast<int64_t>(a.S) + kFlatThreads - 1) / kFlatThreads : 0;
    if (row_blocks + dw_blocks == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(row_blocks + dw_blocks)), block(kFlatThreads);
    if (a.dtype == 1) {
      if (a.dw) combine_bwd_flat_kernel<bf16_t, true, true><<<grid, block, 0, st>>>(a, lg, total, row_blocks);
      else if (lg >= 0) combine_bwd_flat_kernel<bf16_t, true, false><<<grid, block, 0, st>>>(a, lg, total, row_blocks);
      else combine_bwd_flat_kernel<bf16_t, false, false><<<grid, block, 0, st>>>(a, lg, total, row_blocks);
    } else {
      if (a.dw) combine_bwd_flat_kernel<float, true, true><<<grid, block, 0, st>>>(a, lg, total, row_blocks);
      else if (lg >= 0) combine_bwd_flat_kernel<float, true, false><<<grid, block, 0, st>>>(a, lg, total, row_blocks);
      else combine_bwd_flat_kernel<float, false, false><<<grid, block, 0, st>>>(a, lg, total, row_blocks);
    }
    return hipGetLastError();
  }
  const int64_t row_blocks = blocks_for_rows(a.rows, kWideWaves);
  const int64_t dw_blocks = (static_cast<int64_t>(a.S) * a.k + kThreads - 1) / kThreads;
  if (row_blocks + dw_blocks == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(row_blocks + dw_blocks)), block(kThreads);
  if (a.dtype == 1) {
    if (a.dw) combine_bwd_kernel<bf16_t, true><<<grid, block, 0, st>>>(a, row_blocks);
    else combine_bwd_kernel<bf16_t, false><<<grid, block, 0, st>>>(a, row_blocks);
  } else {
    if (a.dw) combine_bwd_kernel<float, true><<<grid, block, 0, st>>>(a, row_blocks);
    else combine_bwd_kernel<float, false><<<grid, block, 0, st>>>(a, row_blocks);
  }
  return hipGetLastError();
}

}  // namespace hetumoe
