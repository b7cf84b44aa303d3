// Layout-transform kernels for gfx950: steps 2 and 6 of Algorithm 1 and their
// gradients.  Every output row has exactly one writer, so there are no atomics
// and results are bitwise reproducible.  Outputs indexed by token (combine,
// dispatch backward) are gathers; outputs indexed by expert slot (dispatch,
// combine backward) are gathers over slots for k = 1 and token-major scatters
// for k > 1, so that each token row is read once from memory.
//
// The kernels are bound by HBM bandwidth, and on MI355X how a kernel writes
// matters as much as how it reads (measured at the hash workload's shape,
// 8 KiB rows, 1 GiB expert buffers, in pass order):
// * Writers of [E,C,d] buffers larger than the Infinity Cache run in two
//   phases of one launch: the first blocks write the empty slots' zero rows,
//   the later blocks the copied rows.  Two pure streams (a fill, then a copy)
//   beat one interleaved stream (dispatch 256 -> 236 us).
// * Writers of token rows (combine, dispatch backward) give a row to a block
//   of threads, one 16-byte chunk each, and store through buffer instructions
//   with an explicit cache policy: rows with data non-temporal at every scope
//   (sc0 sc1 nt), zero rows of tokens with nothing kept sc1 only, which lets
//   those writes merge in the caches (combine 165 -> 156 us).  Plain stores of
//   whole [E,C,d] buffers instead leave dirty lines behind that slow the next
//   kernel, so those writers keep non-temporal stores.
// * Row indices are made wave-uniform (readfirstlane) wherever a wave lies
//   inside one row, so that routing comes through scalar loads and buffer
//   resources sit in scalar registers; a per-lane resource would make the
//   compiler loop over the lanes' distinct values.
// Source rows are read with non-temporal loads: each is read once.
#include "common.hpp"
#include "kernels.hpp"

namespace hetumoe {

constexpr int kUnroll = 8;
constexpr int kWideWaves = 16;  // one row (or token) per wave, 16 waves per block
constexpr int kDispWaves = 4;   // waves per block of the choice-major dispatch (k > 1)
// Waves per block of the choice-major combine backward (k > 1).
constexpr int kBwdScatterWaves = 8;

// Row kernels: kRowThreads threads, one 16-byte chunk each per step.
constexpr int kRowThreads = 512;
constexpr int kRowWaves = kRowThreads / kWave;

// Cache-policy bits of gfx950's buffer instructions (sc0 = 1, nt = 2, sc1 = 16)
// and word 3 of a raw buffer resource of 32-bit elements (gfx9 family).
constexpr int kPolDataRow = 1 | 2 | 16;
constexpr int kPolZeroRow = 16;
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ void store_nt(u32x4* p, const u32x4& v) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ u32x4 load_nt(const u32x4* p) { return __builtin_nontemporal_load(p); }

// Row and column of chunk gb + off of a flattened [rows, nch] output, where gb
// is the block's first chunk (row_b, col_b precomputed).  POW2: nch = 1 << lg.
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

// Buffer-resource helpers.  A resource must sit in scalar registers, so every
// base passed here is uniform over the wave (the block's first chunk, or a
// row index made uniform with readfirstlane where a wave lies inside one row).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, bytes, kRsrcWord3);
}
__device__ __forceinline__ u32x4 buf_load_nt(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);
}
__device__ __forceinline__ void buf_store_nt(const u32x4& v, __amdgpu_buffer_rsrc_t r, int off) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 2);
}

// ---------------------------------------------------------------- [E,C,d] writers, k = 1
// xe[row] = x[slot_src[row]] (dispatch) or dye[row] = w[src] * dy[src] with,
// under DW, dw[src] = <dy[src], ye[row]> (combine backward); zeros for an empty
// slot.  TWO (buffers larger than the 256 MB Infinity Cache): blocks [0, nb)
// take the zero rows of their 512 chunks, blocks [nb, 2 nb) the copied rows of
// the same chunks; otherwise each block takes both kinds of its chunks (a
// buffer the cache holds measured faster written in one pass: workload of
// 32768 tokens at 4 KiB rows, dispatch 38.9 -> 33.3 us).  Blocks past the row
// blocks clear dw of dropped choices.  WR (rows a multiple of 64 chunks): every wave lies inside
// one row, whose index, source and branches are then wave-uniform (scalar
// loads of slot_src, buffer resources per row).  With DW a row is a power of
// two of 64 to 512 chunks, so every row lies inside one block: each wave sums
// its part of the dot product, one thread per row adds its waves' parts in
// order.
template <typename T, bool SCALE, bool DW, bool POW2, bool WR, bool TWO>
__global__ __launch_bounds__(kRowThreads) void slot_rows_kernel(RowArgs a, int lg, int64_t total, int64_t nb) {
  constexpr int kEl = Chunk<T>::kElems;
  const int nch = a.nch, S = a.S;
  const int32_t* slot_src = a.slot_src;
  const u32x4* srcp = reinterpret_cast<const u32x4*>(a.src);
  u32x4* dstp = reinterpret_cast<u32x4*>(a.dst);
  const float* wts = a.weights;
  const int64_t bid = blockIdx.x;
  const int64_t row_grid = TWO ? 2 * nb : nb;
  if (bid >= row_grid) {
    if constexpr (DW) {
      const int64_t i = (bid - row_grid) * kRowThreads + threadIdx.x;
      if (i < a.S && a.slots[i] < 0) a.dw[i] = 0.f;
    }
    return;
  }
  const bool full_phase = !TWO || bid >= nb;
  const int64_t gb = (TWO && full_phase ? bid - nb : bid) * kRowThreads;
  const int64_t row_b = POW2 ? 0 : gb / nch;
  const int col_b = POW2 ? 0 : static_cast<int>(gb - row_b * nch);
  int64_t row;
  int col;
  flat_pos<POW2>(gb, row_b, col_b, static_cast<int>(threadIdx.x), nch, lg, row, col);
  if constexpr (WR) row = __builtin_amdgcn_readfirstlane(static_cast<int>(row));  // rows < 2^31
  const int64_t g = gb + threadIdx.x;
  const bool in = g < total;  // wave-uniform under WR (total is a multiple of 64)
  // entries outside [0, S) are out of contract and treated as empty slots
  const int src = in ? slot_src[row] : -1;
  const bool full = (src >= 0) & (src < S);
  float dot = 0.f;
  if (in && (!TWO || full == full_phase)) {
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    float w = 0.f;
    if (full) {
      const u32x4* srow = srcp + static_cast<int64_t>(src) * nch;
      if constexpr (WR) v = buf_load_nt(buf_rsrc(srow, nch * 16), col * 16);
      else v = load_nt(srow + col);
      if constexpr (SCALE) w = wts[src];
    }
    if constexpr (SCALE) {
      if (full) {
        float f[kEl];
        Chunk<T>::unpack(v, f);
        if constexpr (DW) {
          float gq[kEl];
          const u32x4* yb = reinterpret_cast<const u32x4*>(a.aux) + gb;
          Chunk<T>::unpack(WR ? buf_load_nt(buf_rsrc(yb, kRowThreads * 16), threadIdx.x * 16) : load_nt(yb + threadIdx.x), gq);
#pragma unroll
          for (int q = 0; q < kEl; ++q) dot = fmaf(f[q], gq[q], dot);
        }
#pragma unroll
        for (int q = 0; q < kEl; ++q) f[q] *= w;
        v = Chunk<T>::pack(f);
      }
    }
    u32x4* db = dstp + gb;
    if constexpr (WR) buf_store_nt(v, buf_rsrc(db, kRowThreads * 16), threadIdx.x * 16);
    else store_nt(db + threadIdx.x, v);
  }
  if constexpr (DW) {
    if (!full_phase) return;  // uniform over the block
    __shared__ float part[kRowWaves];
    const float t = wave_sum(dot);
    if (lane_id() == 0) part[threadIdx.x / kWave] = t;
    __syncthreads();
    const int rows_here = kRowThreads >> lg;
    const int parts = nch / kWave;
    if (static_cast<int>(threadIdx.x) < rows_here) {
      const int64_t r = (gb >> lg) + threadIdx.x;
      if (r < a.rows) {
        float sum = 0.f;
        for (int j = 0; j < parts; ++j) sum += part[threadIdx.x * parts + j];
        const int s2 = a.slot_src[r];
        if (s2 >= 0 && s2 < a.S) a.dw[s2] = sum;
      }
    }
  }
}

// The same for rows of NCH = 2^LG chunks, 64 to 512 (one to eight waves, so
// every row lies inside one block), with nothing but the block and phase
// indices on the path to the first load: blockIdx.y is the phase (TWO: 0 zero
// rows, 1 copied rows; else 0 both), chunks past the buffer are clamped onto
// its last one and their stores skipped, and an empty slot or a chunk of the
// other phase skips its load by a branch uniform over the wave.  The first
// phase's blocks below ceil(S / 512) also clear dw of dropped choices.
template <typename T, bool SCALE, bool DW, int LG, bool TWO>
__global__ __launch_bounds__(kRowThreads) void slot_rows_pow2_kernel(RowArgs a, int64_t total) {
  constexpr int kEl = Chunk<T>::kElems;
  constexpr int NCH = 1 << LG;
  const bool copy_phase = !TWO || blockIdx.y == 1;
  const int64_t gb = static_cast<int64_t>(blockIdx.x) * kRowThreads;
  const int64_t g = gb + threadIdx.x;
  const bool live = g < total;
  const int64_t gc = live ? g : total - 1;  // total > 0
  const int row = __builtin_amdgcn_readfirstlane(static_cast<int>(gc >> LG));
  const int col = static_cast<int>(gc & (NCH - 1));
  // entries outside [0, S) are out of contract and treated as empty slots
  const int src = a.slot_src[row];
  const bool full = (src >= 0) & (src < a.S);
  // uniform over the wave: its chunks lie in one row, and total is a multiple of 64
  const bool act = __builtin_amdgcn_readfirstlane(static_cast<int>(live & (!TWO || full == copy_phase))) != 0;
  u32x4 v = u32x4{0u, 0u, 0u, 0u};
  float dot = 0.f;
  if (copy_phase && act && full) {
    const u32x4* srow = reinterpret_cast<const u32x4*>(a.src) + static_cast<int64_t>(src) * NCH;
    v = buf_load_nt(buf_rsrc(srow, NCH * 16), col * 16);
    if constexpr (SCALE) {
      const float w = a.weights[src];
      u32x4 ve = u32x4{0u, 0u, 0u, 0u};
      if constexpr (DW)
        ve = buf_load_nt(buf_rsrc(reinterpret_cast<const u32x4*>(a.aux) + gb, kRowThreads * 16),
                         static_cast<int>(threadIdx.x) * 16);
      {
        float f[kEl];
        Chunk<T>::unpack(v, f);
        if constexpr (DW) {
          float gq[kEl];
          Chunk<T>::unpack(ve, gq);
#pragma unroll
          for (int q = 0; q < kEl; ++q) dot = fmaf(f[q], gq[q], dot);
        }
#pragma unroll
        for (int q = 0; q < kEl; ++q) f[q] *= w;
        v = Chunk<T>::pack(f);
      }
    }
  }
  if (act) buf_store_nt(v, buf_rsrc(reinterpret_cast<u32x4*>(a.dst) + gb, kRowThreads * 16), threadIdx.x * 16);
  if constexpr (DW) {
    if (blockIdx.y == 0) {
      const int64_t i = gb + threadIdx.x;
      if (i < a.S && a.slots[i] < 0) a.dw[i] = 0.f;
    }
    if (!copy_phase) return;  // uniform over the block
    __shared__ float part[kRowWaves];
    const float t = wave_sum(dot);
    if (lane_id() == 0) part[threadIdx.x / kWave] = t;
    __syncthreads();
    constexpr int kRowsHere = kRowThreads / NCH;
    constexpr int kParts = NCH / kWave;
    if (static_cast<int>(threadIdx.x) < kRowsHere) {
      const int64_t r = (gb >> LG) + threadIdx.x;
      if (r < a.rows) {
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < kParts; ++j) sum += part[threadIdx.x * kParts + j];
        const int s2 = a.slot_src[r];
        if (s2 >= 0 && s2 < a.S) a.dw[s2] = sum;
      }
    }
  }
}

// Combine backward with dw for k = 1 on rows slot_rows_kernel does not take
// (not a power of two, or longer than 512 chunks): one wave per row, kUnroll
// chunks per lane in flight.  Blocks past the row blocks clear dw of dropped
// choices.
template <typename T>
__global__ __launch_bounds__(kWideWaves * kWave) void combine_bwd_wave_kernel(RowArgs a, int64_t row_blocks) {
  constexpr int kEl = Chunk<T>::kElems;
  if (static_cast<int64_t>(blockIdx.x) >= row_blocks) {
    const int64_t i = (static_cast<int64_t>(blockIdx.x) - row_blocks) * (kWideWaves * kWave) + threadIdx.x;
    if (i < static_cast<int64_t>(a.S) * a.k && a.slots[i] < 0) a.dw[i] = 0.f;
    return;
  }
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kWideWaves + threadIdx.x / kWave;
  if (row >= a.rows) return;
  const int lane = lane_id();
  const int nch = a.nch;
  const int src = a.slot_src[row];
  u32x4* dst = reinterpret_cast<u32x4*>(a.dst) + row * nch;
  if (src < 0 || src >= a.S * a.k) {  // empty (or out-of-contract) slot
    for (int i = lane; i < nch; i += kWave) store_nt(dst + i, u32x4{0u, 0u, 0u, 0u});
    return;
  }
  const float w = a.weights[src];
  const u32x4* dyrow = reinterpret_cast<const u32x4*>(a.src) + static_cast<int64_t>(src / a.k) * nch;
  const u32x4* yerow = reinterpret_cast<const u32x4*>(a.aux) + row * nch;
  float dot = 0.f;
  for (int base = 0; base < nch; base += kWave * kUnroll) {
    u32x4 v[kUnroll], ve[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = base + u * kWave + lane;
      if (i < nch) {
        v[u] = load_nt(dyrow + i);
        ve[u] = load_nt(yerow + i);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = base + u * kWave + lane;
      if (i < nch) {
        float f[kEl], g[kEl];
        Chunk<T>::unpack(v[u], f);
        Chunk<T>::unpack(ve[u], g);
#pragma unroll
        for (int q = 0; q < kEl; ++q) dot = fmaf(f[q], g[q], dot);
#pragma unroll
        for (int q = 0; q < kEl; ++q) f[q] *= w;
        store_nt(dst + i, Chunk<T>::pack(f));
      }
    }
  }
  dot = wave_sum(dot);
  if (lane == 0) a.dw[src] = dot;
}

// ---------------------------------------------------------------- token rows: combine, dispatch backward
// y[s] = sum_{r kept} w[s,r] * ye[ids[s,r], slots[s,r]]  (WEIGHTED)
// dx[s] = sum_{r kept} dxe[ids[s,r], slots[s,r]]        (!WEIGHTED)
// fp32 accumulation in r order, one rounding to T.  A block takes rpb rows of
// tpr threads (tpr = nch for rows of up to 512 chunks, else 512 threads
// walking the row); a thread loads the chunk of every kept choice before it
// sums them (CPT chunks each, tpr * CPT chunks per row and step: with several
// choices, more loads in flight).  WR (tpr a multiple of 64): the token of a wave is uniform, its
// routing comes through scalar loads, and the row is stored through a buffer
// resource with the cache policy of its kind: kPolDataRow, or kPolZeroRow for
// a token with nothing kept.
template <typename T, bool WEIGHTED, int KMAX, bool WR, int CPT, int TPR>
__global__ __launch_bounds__(kRowThreads) void token_rows_kernel(RowArgs a, int tpr_arg, int rpb_arg) {
  constexpr int kEl = Chunk<T>::kElems;
  // TPR > 0 (then also WR): threads per row known when compiled, a row is
  // exactly TPR * CPT chunks, and every thread of the block has a row.  That
  // path has no branch before its loads: rows past the batch are clamped onto
  // the last one (their stores are skipped), and a dropped choice loads from an
  // offset past its buffer resource, which returns zeros without a memory access.
  const int tpr = TPR > 0 ? TPR : tpr_arg;
  const int rpb = TPR > 0 ? kRowThreads / TPR : rpb_arg;
  const int rl = static_cast<int>(threadIdx.x) / tpr;
  int64_t s = static_cast<int64_t>(blockIdx.x) * rpb + rl;
  const bool live = TPR > 0 ? s < a.rows : (rl < rpb && s < a.rows);
  if constexpr (TPR > 0) {
    if (s >= a.rows) s = a.rows - 1;
  } else if (!live) {
    return;
  }
  if constexpr (WR) s = __builtin_amdgcn_readfirstlane(static_cast<int>(s));  // rows < 2^31
  const int nch = a.nch;
  const int k = KMAX <= 2 ? KMAX : a.k;  // the launcher picks KMAX = k for k <= 2
  const u32x4* src = reinterpret_cast<const u32x4*>(a.src);
  // every routing value is loaded before any is tested, so that the loads
  // overlap (a short-circuit test would make each wait for the one before)
  int slot[KMAX], e[KMAX];
  float w[KMAX];
#pragma unroll
  for (int r = 0; r < KMAX; ++r) {
    const bool have = r < k;
    slot[r] = have ? a.slots[s * k + r] : -1;
    e[r] = have ? a.ids[s * k + r] : 0;
    w[r] = (WEIGHTED && have) ? a.weights[s * k + r] : 1.f;
  }
  int64_t off[KMAX];
  bool ok[KMAX];
  bool any = false;
#pragma unroll
  for (int r = 0; r < KMAX; ++r) {
    // dropped choices (slot -1) and out-of-contract entries contribute nothing
    ok[r] = (slot[r] >= 0) & (slot[r] < a.C) & (e[r] >= 0) & (e[r] < a.E);
    off[r] = ok[r] ? (static_cast<int64_t>(e[r]) * a.C + slot[r]) * nch : 0;
    any = any | ok[r];
  }
  u32x4* orow = reinterpret_cast<u32x4*>(a.dst) + s * nch;
  if constexpr (TPR > 0) {
    const __amdgpu_buffer_rsrc_t out = buf_rsrc(orow, nch * 16);
    const int c0 = static_cast<int>(threadIdx.x) - rl * tpr;
    u32x4 v[CPT][KMAX];
#pragma unroll
    for (int u = 0; u < CPT; ++u)
#pragma unroll
      for (int r = 0; r < KMAX; ++r)
        v[u][r] = buf_load_nt(buf_rsrc(src + off[r], nch * 16), ok[r] ? (c0 + u * tpr) * 16 : 0x7ffffff0);
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      float acc[kEl];
#pragma unroll
      for (int q = 0; q < kEl; ++q) acc[q] = 0.f;
#pragma unroll
      for (int r = 0; r < KMAX; ++r) {
        if (!ok[r]) continue;
        float f[kEl];
        Chunk<T>::unpack(v[u][r], f);
#pragma unroll
        for (int q = 0; q < kEl; ++q) acc[q] = WEIGHTED ? fmaf(w[r], f[q], acc[q]) : acc[q] + f[q];
      }
      const u32x4 o = Chunk<T>::pack(acc);
      if (live) {
        if (any) __builtin_amdgcn_raw_buffer_store_b128(o, out, (c0 + u * tpr) * 16, 0, kPolDataRow);
        else __builtin_amdgcn_raw_buffer_store_b128(o, out, (c0 + u * tpr) * 16, 0, kPolZeroRow);
      }
    }
    return;
  }
  for (int c0 = static_cast<int>(threadIdx.x) - rl * tpr; c0 < nch; c0 += tpr * CPT) {
    u32x4 v[CPT][KMAX];
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const int c = c0 + u * tpr;
#pragma unroll
      for (int r = 0; r < KMAX; ++r) {
        if (!ok[r] || c >= nch) continue;
        if constexpr (WR) v[u][r] = buf_load_nt(buf_rsrc(src + off[r], nch * 16), c * 16);
        else v[u][r] = load_nt(src + off[r] + c);
      }
    }
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const int c = c0 + u * tpr;
      if (c >= nch) continue;
      float acc[kEl];
#pragma unroll
      for (int q = 0; q < kEl; ++q) acc[q] = 0.f;
#pragma unroll
      for (int r = 0; r < KMAX; ++r) {
        if (!ok[r]) continue;
        float f[kEl];
        Chunk<T>::unpack(v[u][r], f);
#pragma unroll
        for (int q = 0; q < kEl; ++q) acc[q] = WEIGHTED ? fmaf(w[r], f[q], acc[q]) : acc[q] + f[q];
      }
      const u32x4 o = Chunk<T>::pack(acc);
      if constexpr (WR) {
        const __amdgpu_buffer_rsrc_t out = buf_rsrc(orow, nch * 16);
        if (any) __builtin_amdgcn_raw_buffer_store_b128(o, out, c * 16, 0, kPolDataRow);
        else __builtin_amdgcn_raw_buffer_store_b128(o, out, c * 16, 0, kPolZeroRow);
      } else {
        store_nt(orow + c, o);
      }
    }
  }
}

// ---------------------------------------------------------------- token-major forms (k > 1)
// With several choices per token, the slot-major gathers above read each token
// row once per kept choice, at times far apart.  These forms walk the choices
// in token order instead: one choice per wave, the choices of a token side by
// side, so that the token row comes from memory once.  The
// remaining blocks stride over the expert slots and zero the empty ones.  Each
// output row still has exactly one writer.
constexpr int kZeroBlocks = 1024;

// first_wave is uniform over the wave (made so by the callers), so the rows,
// their slot_src entries and the buffer resources are too.
__device__ __forceinline__ void zero_empty_rows(const RowArgs& a, int first_wave, int64_t nwaves, int lane) {
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (int64_t row = first_wave; row < a.rows; row += nwaves) {
    const int src = a.slot_src[row];
    if (src >= 0 && src < a.S * a.k) continue;
    const __amdgpu_buffer_rsrc_t dst = buf_rsrc(reinterpret_cast<u32x4*>(a.dst) + row * a.nch, a.nch * 16);
    for (int i = lane; i < a.nch; i += kWave) buf_store_nt(z, dst, i * 16);
  }
}

// xe[ids[s,r], slots[s,r]] = x[s] for every kept (s, r); empty slots zero.
// One wave per choice (s, r), the k waves of a token next to each other in a
// block: x[s] comes from memory for the first and from the L2 for the others
// (cached loads).  A wave per token writing its k rows in turn measured slower
// (workload of 32768 tokens, k = 4, 4 KiB rows, with drops: 168 -> 125 us).
__global__ __launch_bounds__(kDispWaves * kWave) void dispatch_scatter_kernel(RowArgs a, int64_t pair_blocks) {
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  if (static_cast<int64_t>(blockIdx.x) >= pair_blocks) {
    zero_empty_rows(a, __builtin_amdgcn_readfirstlane(
                           static_cast<int>((static_cast<int64_t>(blockIdx.x) - pair_blocks) * kDispWaves + wave)),
                    static_cast<int64_t>(gridDim.x - pair_blocks) * kDispWaves, lane);
    return;
  }
  // the choice is uniform over the wave: scalar routing loads, row resources in
  // scalar registers; chunks past the row fall outside its resource (loads give
  // zeros, stores are dropped), so the row walk needs no bounds test
  const int64_t pr = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<int64_t>(blockIdx.x) * kDispWaves + wave));
  if (pr >= static_cast<int64_t>(a.S) * a.k) return;
  const int slot = a.slots[pr];
  const int e = a.ids[pr];
  if (!((slot >= 0) & (slot < a.C) & (e >= 0) & (e < a.E))) return;
  const int nch = a.nch;
  const int64_t s = pr / a.k;
  const int64_t row = static_cast<int64_t>(e) * a.C + slot;
  const __amdgpu_buffer_rsrc_t srow = buf_rsrc(reinterpret_cast<const u32x4*>(a.src) + s * nch, nch * 16);
  const __amdgpu_buffer_rsrc_t dst = buf_rsrc(reinterpret_cast<u32x4*>(a.dst) + row * nch, nch * 16);
  for (int base = 0; base < nch; base += kWave * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_amdgcn_raw_buffer_load_b128(srow, (base + u * kWave + lane) * 16, 0, 0);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) buf_store_nt(v[u], dst, (base + u * kWave + lane) * 16);
  }
}

// For every kept (s, r): dye[ids, slots] = w[s,r] * dy[s] and, with DW,
// dw[s,r] = <dy[s], ye[ids, slots]>; dropped choices get dw = 0; empty slots
// of dye are zero.  One wave per choice (s, r), the k waves of a token next to
// each other in a block: dy[s] comes from memory for the first of them and
// from the L2 for the others (cached loads), each ye row is read once
// (non-temporal).  A wave per token carrying all k dot products held ~126
// VGPRs; a wave per choice holds ~72 (workload of 32768 tokens, k = 4, 4 KiB
// rows: 235 -> 207 us).
template <typename T, bool DW>
__global__ __launch_bounds__(kBwdScatterWaves * kWave) void combine_bwd_scatter_kernel(RowArgs a, int64_t pair_blocks) {
  constexpr int kEl = Chunk<T>::kElems;
  constexpr int kU = 4;  // chunks per lane per step
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  if (static_cast<int64_t>(blockIdx.x) >= pair_blocks) {
    zero_empty_rows(a, __builtin_amdgcn_readfirstlane(
                           static_cast<int>((static_cast<int64_t>(blockIdx.x) - pair_blocks) * kBwdScatterWaves + wave)),
                    static_cast<int64_t>(gridDim.x - pair_blocks) * kBwdScatterWaves, lane);
    return;
  }
  // the choice is uniform over the wave (scalar routing, row resources in
  // scalar registers); chunks past a row fall outside its resource: loads give
  // zeros, stores are dropped, so the row walk needs no bounds test
  const int64_t pr = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<int64_t>(blockIdx.x) * kBwdScatterWaves + wave));
  if (pr >= static_cast<int64_t>(a.S) * a.k) return;
  const int slot = a.slots[pr];
  const int e = a.ids[pr];
  if (!((slot >= 0) & (slot < a.C) & (e >= 0) & (e < a.E))) {
    if constexpr (DW)
      if (lane == 0) a.dw[pr] = 0.f;
    return;
  }
  const int nch = a.nch;
  const int64_t s = pr / a.k;
  const int64_t row = static_cast<int64_t>(e) * a.C + slot;
  const float w = a.weights[pr];
  const __amdgpu_buffer_rsrc_t dyrow = buf_rsrc(reinterpret_cast<const u32x4*>(a.src) + s * nch, nch * 16);
  const __amdgpu_buffer_rsrc_t dst = buf_rsrc(reinterpret_cast<u32x4*>(a.dst) + row * nch, nch * 16);
  float dot = 0.f;
  for (int base = 0; base < nch; base += kWave * kU) {
    u32x4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) v[u] = __builtin_amdgcn_raw_buffer_load_b128(dyrow, (base + u * kWave + lane) * 16, 0, 0);
    u32x4 g[DW ? kU : 1];
    if constexpr (DW) {
      const __amdgpu_buffer_rsrc_t yerow = buf_rsrc(reinterpret_cast<const u32x4*>(a.aux) + row * nch, nch * 16);
#pragma unroll
      for (int u = 0; u < kU; ++u) g[u] = buf_load_nt(yerow, (base + u * kWave + lane) * 16);
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      float f[kEl];
      Chunk<T>::unpack(v[u], f);
      if constexpr (DW) {
        float gq[kEl];
        Chunk<T>::unpack(g[u], gq);
#pragma unroll
        for (int q = 0; q < kEl; ++q) dot = fmaf(f[q], gq[q], dot);
      }
#pragma unroll
      for (int q = 0; q < kEl; ++q) f[q] *= w;
      buf_store_nt(Chunk<T>::pack(f), dst, (base + u * kWave + lane) * 16);
    }
  }
  if constexpr (DW) {
    const float t = wave_sum(dot);
    if (lane == 0) a.dw[pr] = t;
  }
}

// ---------------------------------------------------------------- launchers
// log2(n) for a power of two, else -1
static inline int pow2_log(int n) {
  if (n <= 0 || (n & (n - 1)) != 0) return -1;
  int lg = 0;
  while ((1 << lg) < n) ++lg;
  return lg;
}

static inline int64_t row_blocks(int64_t total) { return (total + kRowThreads - 1) / kRowThreads; }

// Output size above which the [E,C,d] writers run in two phases (the Infinity
// Cache of MI355X holds 256 MB).
constexpr int64_t kTwoPhaseBytes = int64_t(256) << 20;

template <typename T, bool SCALE, bool DW, bool TWO>
static void launch_slot_rows_t(const RowArgs& a, int64_t total, int64_t nb, hipStream_t st) {
  const int64_t dwb = DW ? (static_cast<int64_t>(a.S) + kRowThreads - 1) / kRowThreads : 0;
  const unsigned grid = static_cast<unsigned>((TWO ? 2 * nb : nb) + dwb);
  if (grid == 0) return;
  const int lg = pow2_log(a.nch);
  const dim3 g(grid), block(kRowThreads);
  if (a.nch % kWave == 0) {
    if (lg >= 0) slot_rows_kernel<T, SCALE, DW, true, true, TWO><<<g, block, 0, st>>>(a, lg, total, nb);
    else slot_rows_kernel<T, SCALE, DW, false, true, TWO><<<g, block, 0, st>>>(a, lg, total, nb);
  } else {
    if (lg >= 0) slot_rows_kernel<T, SCALE, DW, true, false, TWO><<<g, block, 0, st>>>(a, lg, total, nb);
    else slot_rows_kernel<T, SCALE, DW, false, false, TWO><<<g, block, 0, st>>>(a, lg, total, nb);
  }
}

template <typename T, bool SCALE, bool DW, int LG>
static void launch_slot_rows_pow2(const RowArgs& a, int64_t total, hipStream_t st) {
  const int64_t nb = row_blocks(total);
  const int64_t dwb = DW ? (static_cast<int64_t>(a.S) + kRowThreads - 1) / kRowThreads : 0;
  const dim3 block(kRowThreads);
  if (total * 16 > kTwoPhaseBytes) {
    slot_rows_pow2_kernel<T, SCALE, DW, LG, true>
        <<<dim3(static_cast<unsigned>(nb > dwb ? nb : dwb), 2), block, 0, st>>>(a, total);
  } else {
    slot_rows_pow2_kernel<T, SCALE, DW, LG, false>
        <<<dim3(static_cast<unsigned>(nb > dwb ? nb : dwb), 1), block, 0, st>>>(a, total);
  }
}

template <typename T, bool SCALE, bool DW>
static void launch_slot_rows(const RowArgs& a, hipStream_t st) {
  const int64_t total = a.rows * a.nch;
  const int lg = pow2_log(a.nch);
  if (total > 0 && lg >= 6 && lg <= 9) {
    if (lg == 9) launch_slot_rows_pow2<T, SCALE, DW, 9>(a, total, st);
    else if (lg == 8) launch_slot_rows_pow2<T, SCALE, DW, 8>(a, total, st);
    else if (lg == 7) launch_slot_rows_pow2<T, SCALE, DW, 7>(a, total, st);
    else launch_slot_rows_pow2<T, SCALE, DW, 6>(a, total, st);
    return;
  }
  const int64_t nb = row_blocks(total);
  if (total * 16 > kTwoPhaseBytes) launch_slot_rows_t<T, SCALE, DW, true>(a, total, nb, st);
  else launch_slot_rows_t<T, SCALE, DW, false>(a, total, nb, st);
}

static unsigned zero_blocks(int64_t rows, int waves) {
  const int64_t b = (rows + waves - 1) / waves;
  const int64_t cap = static_cast<int64_t>(kZeroBlocks) * kWideWaves / waves;
  return static_cast<unsigned>(b < cap ? b : cap);
}

hipError_t launch_dispatch(const RowArgs& a, hipStream_t st) {
  if (a.k > 1) {
    const int64_t pair_blocks = (static_cast<int64_t>(a.S) * a.k + kDispWaves - 1) / kDispWaves;
    const unsigned grid = static_cast<unsigned>(pair_blocks) + zero_blocks(a.rows, kDispWaves);
    if (grid == 0) return hipSuccess;
    dispatch_scatter_kernel<<<dim3(grid), dim3(kDispWaves * kWave), 0, st>>>(a, pair_blocks);
    return hipGetLastError();
  }
  // the element type is irrelevant to a bit copy
  launch_slot_rows<float, false, false>(a, st);
  return hipGetLastError();
}

template <typename T, bool WEIGHTED, bool WR, int CPT, int TPR>
static void launch_token_rows_k(const RowArgs& a, int tpr, int rpb, hipStream_t st) {
  const dim3 grid(static_cast<unsigned>((a.rows + rpb - 1) / rpb)), block(kRowThreads);
  if (a.k == 1) token_rows_kernel<T, WEIGHTED, 1, WR, CPT, TPR><<<grid, block, 0, st>>>(a, tpr, rpb);
  else if (a.k == 2) token_rows_kernel<T, WEIGHTED, 2, WR, CPT, TPR><<<grid, block, 0, st>>>(a, tpr, rpb);
  else if (a.k <= 4) token_rows_kernel<T, WEIGHTED, 4, WR, CPT, TPR><<<grid, block, 0, st>>>(a, tpr, rpb);
  else token_rows_kernel<T, WEIGHTED, 8, WR, CPT, TPR><<<grid, block, 0, st>>>(a, tpr, rpb);
}

template <typename T, bool WEIGHTED, bool WR, int CPT>
static void launch_token_rows_w(const RowArgs& a, int tpr, int rpb, hipStream_t st) {
  // rows of exactly tpr * CPT chunks with tpr dividing the block: the
  // compile-time path
  const bool exact = WR && a.nch == tpr * CPT;
  if (exact && tpr == 512) launch_token_rows_k<T, WEIGHTED, WR, CPT, 512>(a, tpr, rpb, st);
  else if (exact && tpr == 256) launch_token_rows_k<T, WEIGHTED, WR, CPT, 256>(a, tpr, rpb, st);
  else if (exact && tpr == 128) launch_token_rows_k<T, WEIGHTED, WR, CPT, 128>(a, tpr, rpb, st);
  else launch_token_rows_k<T, WEIGHTED, WR, CPT, 0>(a, tpr, rpb, st);
}

template <typename T, bool WEIGHTED>
static void launch_token_rows_t(const RowArgs& a, hipStream_t st) {
  // with three or more choices, two chunks per thread where rows split evenly
  // into waves; otherwise one
  const int cpt = (a.k >= 3 && a.nch % (2 * kWave) == 0) ? 2 : 1;
  const int rt = a.nch / cpt;  // threads a row would take
  const int tpr = rt <= kRowThreads ? rt : kRowThreads;
  const int rpb = rt <= kRowThreads ? kRowThreads / rt : 1;
  if (cpt == 2) launch_token_rows_w<T, WEIGHTED, true, 2>(a, tpr, rpb, st);
  else if (tpr % kWave == 0) launch_token_rows_w<T, WEIGHTED, true, 1>(a, tpr, rpb, st);
  else launch_token_rows_w<T, WEIGHTED, false, 1>(a, tpr, rpb, st);
}

hipError_t launch_combine(const RowArgs& a, bool weighted, hipStream_t st) {
  if (a.rows == 0 || a.nch == 0) return hipSuccess;
  if (a.dtype == 1) {
    if (weighted) launch_token_rows_t<bf16_t, true>(a, st);
    else launch_token_rows_t<bf16_t, false>(a, st);
  } else {
    if (weighted) launch_token_rows_t<float, true>(a, st);
    else launch_token_rows_t<float, false>(a, st);
  }
  return hipGetLastError();
}

hipError_t launch_combine_bwd(const RowArgs& a, hipStream_t st) {
  if (a.k > 1) {
    const int64_t pair_blocks = (static_cast<int64_t>(a.S) * a.k + kBwdScatterWaves - 1) / kBwdScatterWaves;
    const unsigned grid = static_cast<unsigned>(pair_blocks) + zero_blocks(a.rows, kBwdScatterWaves);
    if (grid == 0) return hipSuccess;
    const dim3 g(grid), block(kBwdScatterWaves * kWave);
    if (a.dtype == 1) {
      if (a.dw) combine_bwd_scatter_kernel<bf16_t, true><<<g, block, 0, st>>>(a, pair_blocks);
      else combine_bwd_scatter_kernel<bf16_t, false><<<g, block, 0, st>>>(a, pair_blocks);
    } else {
      if (a.dw) combine_bwd_scatter_kernel<float, true><<<g, block, 0, st>>>(a, pair_blocks);
      else combine_bwd_scatter_kernel<float, false><<<g, block, 0, st>>>(a, pair_blocks);
    }
    return hipGetLastError();
  }
  // k = 1: two-phase slot rows, with dw where a row is a power of two of 64 to
  // 512 chunks (else one wave per row)
  const int lg = pow2_log(a.nch);
  if (!a.dw) {
    if (a.dtype == 1) launch_slot_rows<bf16_t, true, false>(a, st);
    else launch_slot_rows<float, true, false>(a, st);
    return hipGetLastError();
  }
  if (lg >= 6 && a.nch <= kRowThreads) {
    if (a.dtype == 1) launch_slot_rows<bf16_t, true, true>(a, st);
    else launch_slot_rows<float, true, true>(a, st);
    return hipGetLastError();
  }
  constexpr int kThreads = kWideWaves * kWave;
  const int64_t rb = (a.rows + kWideWaves - 1) / kWideWaves;
  const int64_t dwb = (static_cast<int64_t>(a.S) * a.k + kThreads - 1) / kThreads;
  if (rb + dwb == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(rb + dwb)), block(kThreads);
  if (a.dtype == 1) combine_bwd_wave_kernel<bf16_t><<<grid, block, 0, st>>>(a, rb);
  else combine_bwd_wave_kernel<float><<<grid, block, 0, st>>>(a, rb);
  return hipGetLastError();
}

}  // namespace hetumoe
