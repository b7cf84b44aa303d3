// Argument blocks and launchers of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hetumoe {

struct RouteArgs {
  int S, d, E, k, nb;
  int kind, normalize, logits_in, dtype;
  uint64_t hash_seed;
  const void* x;            // [S, d]
  const void* wg;           // [d, E]
  const float* bias;        // [E] or null
  const int32_t* token_ids; // [S] (hash)
  const int32_t* hash_table; // [hash_vocab] (hash with a table) or null
  int hash_vocab;
  float* logits;            // [S, E]: input (logits_in), output, or null
  int32_t* ids;             // [S, k]
  float* weights;           // [S, k]
  int32_t* hist;            // [k, E, nb] workspace (nb = 64-token wave blocks)
  // the extended gates, for a route kernel that selects on final logits itself
  // (route_fuses_extended): kind 3 is the hierarchical top-k over `groups`
  // groups; temperature > 0 selects on (logits + noise) / temperature
  int groups;
  float temperature;
  const float* noise;       // [S, E] or null
};

struct ScanArgs {
  int E, k, nb, C;
  int32_t* hist;     // [k, E, nb]: counts in, exclusive offsets out
  int32_t* counts;   // [E]
  int32_t* demand;   // [E] or null
  int32_t* slot_src; // [E, C]
};

struct AssignArgs {
  int S, E, k, nb, C;
  const int32_t* ids;  // [S, k]
  const int32_t* offs; // [k, E, nb]
  int32_t* slots;      // [S, k]
  int32_t* slot_src;   // [E, C]
};

struct RowArgs {
  int64_t rows;        // rows processed by the row kernels
  int nch;             // 16-byte chunks per row
  int S, E, k, C, dtype;
  const void* src;     // gather source rows
  const void* aux;     // second source (ye for dw), or null
  const int32_t* ids;
  const int32_t* slots;
  const int32_t* slot_src;
  const float* weights;
  void* dst;
  float* dw;
};

hipError_t launch_route(const RouteArgs& a, hipStream_t st);

// Selection on logits that first take noise and a temperature (Dense-To-Sparse)
// and/or the hierarchical top-k: one block per 64-token wave block.
struct SelectArgs {
  int S, E, k, nb, kind, normalize, groups;
  float temperature;       // > 0: fin = (raw + noise) / temperature; 0: fin = raw
  const float* raw;        // [S, E] logits as projected (or given)
  const float* noise;      // [S, E] or null
  float* fin;              // [S, E] logits the selection uses (may be raw itself)
  int32_t* ids;            // [S, k]
  float* weights;          // [S, k]
  int32_t* hist;           // [k, E, nb]
};
hipError_t launch_select_ext(const SelectArgs& a, hipStream_t st);
hipError_t launch_route_valu_f32(const RouteArgs& a, hipStream_t st);
hipError_t launch_route_valu_bf16(const RouteArgs& a, hipStream_t st);
hipError_t launch_route_mfma(const RouteArgs& a, hipStream_t st);
bool route_uses_mfma(const RouteArgs& a);
hipError_t launch_route_mfma_rs(const RouteArgs& a, int cus, hipStream_t st);
hipError_t launch_route_mfma_ph(const RouteArgs& a, int cus, hipStream_t st);
bool route_uses_mfma_ph(const RouteArgs& a);
// Compute units of the current device (queried once per device).
int device_cu_count();
bool route_uses_mfma_rs(const RouteArgs& a);
// True when the register-resident route kernel takes this projection: it then
// also applies the noise and temperature and the hierarchical top-k itself, so
// the extended gates need no logits round trip.
bool route_fuses_extended(const RouteArgs& a);
hipError_t launch_scan(const ScanArgs& a, hipStream_t st);
hipError_t launch_assign(const AssignArgs& a, hipStream_t st);
// Scan and assign, in one launch when the histogram is small (the offsets then
// stay out of the histogram, which is left as the counts).
hipError_t launch_scan_assign(const ScanArgs& sa, const AssignArgs& a, hipStream_t st);
hipError_t launch_dispatch(const RowArgs& a, hipStream_t st);
hipError_t launch_combine(const RowArgs& a, bool weighted, hipStream_t st);
hipError_t launch_combine_bwd(const RowArgs& a, hipStream_t st);

// Gate backward (gradient of the gate of Eq. 1).  Buffers of the workspace are
// carved out by the C ABI.
struct GateBwdArgs {
  int S, d, E, k, nb;       // nb: 64-token wave blocks
  int kind, normalize, dtype, accumulate;
  float aux_coef;
  float temperature;        // > 0: the logits are (L + noise) / temperature; gradients w.r.t. L
  int nsplit, split_tokens; // dW is summed over tokens in nsplit ranges of split_tokens (a multiple of 64)
  int mfma_dw, mfma_dx;     // matrix-core paths (bf16, E a multiple of 16 up to 128, d a multiple of 64)
  int sums_in_reduce;       // db, the softmax sums and the loss run as extra blocks of the dW reduction
  int64_t s_pad;            // row length of dlt: S rounded up to 64
  const void* x;            // [S, d]
  const void* wg;           // [d, E]
  const float* logits;      // [S, E]
  const int32_t* ids;       // [S, k]
  const float* dw;          // [S, k]
  float* dl;                // [S, E] dL (caller's dlogits or workspace)
  uint16_t* dlt;            // [3][E, s_pad] dL transposed, split into three bf16 planes
                            // (hi + mid + lo == dL), zero beyond S (matrix-core dW only)
  void* dx;                 // [S, d] or null
  float* dwg;               // [d, E] or null
  float* dbias;             // [E] or null
  float* aux_loss;          // [1] or null
  int32_t* cnt;             // [E] first-choice counts (load-balancing loss)
  float* ppart;             // [nb, E] per wave block sums of the softmax (load-balancing loss)
  float* bpart;             // [nb, E] per wave block sums of dL (db)
  float* pe;                // [E] sums of the softmax over all tokens
  float* wpart;             // [nsplit, E, d] partial dW
};

// Matrix-core paths of the gate backward for this shape.
inline bool gate_bwd_mfma_shape(int dtype, int E, int d) {
  return dtype == 1 && E % 16 == 0 && E <= 128 && d % 64 == 0;
}

hipError_t launch_gate_bwd_dl(const GateBwdArgs& a, hipStream_t st);
hipError_t launch_gate_bwd_dwg(const GateBwdArgs& a, hipStream_t st);
hipError_t launch_gate_bwd_dx(const GateBwdArgs& a, hipStream_t st);

// BASE layer gate: balanced assignment by an auction on fp32 scores [S, E]
// (every expert takes exactly cap = S / E tokens).  Buffers of the workspace
// are carved out by the C ABI.
constexpr int kBaseCand = 2048;          // bidders an expert considers per round
constexpr int kBaseMaxCap = 2048;        // largest S / E
constexpr double kBaseEpsStep = 32.0;    // eps divisor between phases
constexpr double kBaseEpsEnd = 0x1p-30;  // final eps, relative to the score range
constexpr int kBaseRangeBlocks = 256;    // blocks of the score-range reduction
constexpr int kBaseTail = 64;            // rounds with at most this many bidders run in one workgroup

// Auction control, double-buffered by round parity (device memory).
struct BaseState {
  double eps, eps_end;     // eps of the current phase, of the last phase
  int phase, rounds_phase, rounds_total;
  int done;                // the auction has ended (converged or failed)
  int failed;              // 1: a phase reached max_rounds; 2: a score is NaN or infinite
  int pad;
};

struct BaseArgs {
  int S, E, cap, nb;       // nb: 64-token wave blocks
  int max_rounds;          // per phase
  const float* logits;     // [S, E]
  double* price;           // [E]
  double* hold_v;          // [E, cap] bids of each expert's holders, best first
  int32_t* hold_t;         // [E, cap] their tokens
  int32_t* hold_n;         // [E]
  int32_t* assign;         // [S] expert of each token, -1 = unassigned
  int32_t* bid_e;          // [S] expert bid for this round, -1 = none
  double* bid_v;           // [S]
  int32_t* bid_cnt;        // [E] bidders of each expert this round
  int32_t* blist;          // [S] this round's bidders, in any order (counts[r & 1] of them)
  int32_t* counts;         // [4] unassigned tokens at the start of a round, by round parity;
                           //     then slots its resolve step filled (kept bidders less evicted holders)
  BaseState* state;        // [2]
  float* range_part;       // [3, kBaseRangeBlocks] per-block min, max, NaN/inf flag
  int32_t* ids;            // [S]
  float* weights;          // [S]
  int32_t* hist;           // [E, nb]
  double* prices_out;      // [E] or null: final prices
  struct BaseHostFlag* host_flag;  // or null: progress written to host memory for the host's pacing
};

// Progress of the synchronous auction, written by the device to pinned host
// memory (system scope) and polled by the host that enqueues the rounds.
struct BaseHostFlag {
  int32_t round;           // last round whose resolve step has started
  int32_t done;            // the auction has ended (converged or failed)
};

struct BaseStats {
  int phases, rounds;      // phases run, rounds summed over phases
  double eps;              // eps of the last phase
  int not_converged;       // a phase reached max_rounds
  int bad_scores;          // a score is infinite or NaN
};

// What the auction did, written to device memory by the asynchronous form
// (the layout of moe_base_status).
struct BaseDevStatus {
  int32_t phases, rounds;  // phases run, rounds summed over phases
  double eps;              // eps of the last phase
  int32_t status;          // 0 converged, 1 not converged within the rounds enqueued or allowed, 2 bad scores
  int32_t pad;
};

size_t base_resolve_lds(int cap);
// Runs the auction and writes ids, weights and hist.  Synchronizes `st`.
hipError_t run_base_auction(const BaseArgs& a, hipStream_t st, BaseStats* stats);
// The same auction with `launch_rounds` rounds enqueued and no host
// synchronization (rounds after the end return at once); the outcome goes to
// `status` in device memory, and every token gets a valid expert even when the
// auction did not finish (its current one, else s mod E).
hipError_t run_base_auction_async(const BaseArgs& a, int launch_rounds, BaseDevStatus* status, hipStream_t st);

}  // namespace hetumoe
