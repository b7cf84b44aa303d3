/*
 * hetumoe.h -- C ABI of the single-GPU MoE gate / layout-transform hot path
 * (HetuMoE, arXiv 2203.14685), built for AMD Instinct MI355X (gfx950).
 *
 * The calls follow Algorithm 1 of the paper (one training step of an MoE layer):
 *   step 1  W, id = Gate(x)                      -> moe_gate
 *   step 2  x' = Layout_Transform(x, id)         -> moe_dispatch
 *   step 6  y = Reverse_Layout_Transform(y', id) -> moe_combine (gate-weighted)
 * plus the gradients of steps 2 and 6            -> moe_dispatch_bwd, moe_combine_bwd,
 * and of step 1                                  -> moe_gate_bwd.
 * Steps 3-5 (AllToAll and the expert networks) are outside this library.
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory     Every buffer argument is DEVICE memory owned by the caller.  Only
 *            the parameter structs are host memory, read during the call.  The
 *            library allocates nothing and keeps no state between calls; it is
 *            reentrant (moe_gate_noalloc alone uses a fixed device array of the
 *            library's, see there).
 * Layout     Row-major, densely packed.  x, y, dy, dx: [S, d].  Expert buffers
 *            xe, ye, dxe, dye: [E, C, d].  Per-choice arrays ids, slots,
 *            weights, dw: [S, k].  logits: [S, E] fp32.  slot_src: [E, C].
 * Dtype      One dtype (fp32 or bf16) for x, Wg and every [S,d] / [E,C,d]
 *            buffer; logits, weights and dw are always fp32; indices int32.
 *            bf16 outputs are rounded once, to nearest-even, from fp32
 *            accumulators.
 * Alignment  [S,d] and [E,C,d] buffers must be 16-byte aligned and rows must be
 *            a multiple of 16 bytes (d * sizeof(elt) % 16 == 0); otherwise the
 *            call returns MOE_ERR_UNSUPPORTED.  Other buffers need their natural
 *            (4-byte) alignment.
 * Async      Each call enqueues its kernels on `stream` (NULL = the default
 *            stream) and returns without waiting.  Nothing is read back to the
 *            host (except by moe_base_gate, which synchronizes its stream).
 *            Outputs must not alias inputs.
 * Outputs    Every output element is overwritten: empty expert slots become zero
 *            rows, unused slot_src entries -1, dropped dw entries 0.
 * Errors     All argument checks run before the first HIP call; a failed check
 *            enqueues nothing.  HIP failures return MOE_ERR_HIP.  A thread-local
 *            message describing the last failure is available from
 *            moe_last_error().  No C++ exception crosses this boundary.
 * Determinism  Results are bitwise reproducible for identical inputs; no
 *            floating-point atomics are used.
 * Range      0 <= S, S*k < 2^31;  1 <= E <= 1024;  0 <= C, E*C < 2^31;  d >= 1.
 *            TOPK: 1 <= k <= min(E, 8).  KTOP1: 1 <= k <= 8 and E % k == 0.
 *            HASH: k == 1.  HTOPK: E % groups == 0, 1 <= k <= min(E / groups, 8).
 *            BASE: S % E == 0, S / E <= 2048.
 */
#ifndef HETUMOE_H
#define HETUMOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_ABI_VERSION 8

/* Symbols of the C ABI are the only ones the shared library exports. */
#define MOE_API __attribute__((visibility("default")))

typedef enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = 1, /* a size, pointer or option is out of the contract */
  MOE_ERR_UNSUPPORTED = 2, /* valid request the library does not handle (alignment, row size) */
  MOE_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than moe_gate_workspace_size() */
  MOE_ERR_HIP = 4,         /* a HIP runtime call failed; see moe_last_error() */
  MOE_ERR_NOT_CONVERGED = 5 /* moe_base_gate: the auction reached its round limit */
} moe_status;

typedef enum { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype;

/* Gating strategies of Sec. 3.1 that share the capacity / layout machinery. */
typedef enum {
  MOE_GATE_TOPK = 0,  /* Top-k of Eq. 1 (Switch: k=1, GShard: k=2) */
  MOE_GATE_KTOP1 = 1, /* kTop1 / expert prototyping: k contiguous groups of E/k experts, top-1 in each */
  MOE_GATE_HASH = 2,  /* Hash Layer: SplitMix64 hash of the token id or a lookup table; k=1, weight 1 */
  MOE_GATE_HTOPK = 3  /* hierarchical top-k (H Topk / SAM): the group holding the best expert, then
                         the k best experts inside that group */
} moe_gate_kind;

/* Parameters of moe_gate (host memory). */
typedef struct {
  int32_t S;          /* tokens */
  int32_t d;          /* model width (row length of x) */
  int32_t E;          /* experts */
  int32_t k;          /* choices per token: experts (TOPK), groups (KTOP1), 1 (HASH) */
  int32_t capacity;   /* C: slots per expert; assignments beyond it are dropped */
  int32_t kind;       /* moe_gate_kind */
  int32_t normalize;  /* TOPK only: 1 = softmax over the k chosen logits (Eq. 1);
                         0 = full softmax over all E, read at each chosen expert (Switch) */
  int32_t logits_in;  /* TOPK/KTOP1: 1 = `logits` is an input (final, bias included), the
                         projection is skipped and x, wg, bias must be NULL;
                         0 = logits are computed from x and wg (+ bias) */
  int32_t dtype;      /* moe_dtype of x and wg */
  int32_t groups;     /* HTOPK: number of contiguous expert groups of E / groups; 0 for other kinds */
  uint64_t hash_seed; /* HASH only: seed of the SplitMix64 hash */
  float temperature;  /* TOPK/KTOP1/HTOPK, Dense-To-Sparse: > 0 makes the gate act on
                         (L + noise) / temperature; 0 = plain logits (noise must be NULL) */
  int32_t hash_vocab; /* HASH: length of hash_table (ids are hash_table[token_id]); 0 = SplitMix64 */
} moe_gate_params;

/* Shape of a dispatch / combine call (host memory). */
typedef struct {
  int32_t S, d, E, k, capacity;
  int32_t dtype; /* moe_dtype of every [S,d] and [E,C,d] buffer */
} moe_layout;

/* Bytes of device workspace moe_gate needs for `p` (0 is possible).  Fails with
 * MOE_ERR_INVALID_ARG for parameters moe_gate would reject. */
MOE_API moe_status moe_gate_workspace_size(const moe_gate_params* p, size_t* bytes);

/*
 * moe_gate -- step 1 of Algorithm 1: the gate network, plus the capacity rule
 * of Sec. 3.1 (capacity factor caps the tokens each expert receives).
 *
 * Computes, per token s:
 *   logits  L[s,e] = sum_j x[s,j] * wg[j,e] + bias[e]     (x . W of Eq. 1; fp32 accumulation)
 *           with temperature > 0 (Dense-To-Sparse gate, Sec. 3.1): L = (L + noise[s,e]) / temperature,
 *           one fp32 addition and one correctly rounded fp32 division; noise (a Gumbel sample,
 *           drawn by the caller) may be NULL
 *   ids     TOPK : the k experts with the largest logits, best first;
 *           KTOP1: the best expert of each group g, [g*E/k, (g+1)*E/k);
 *           HTOPK: with groups of G = E/groups contiguous experts, the group holding the best
 *                  expert, then the k best experts of that group (Sec. 3.1, H Topk);
 *           HASH : hash_table[token_ids[s]] when hash_vocab > 0 (Hash Layer balanced
 *                  assignment, see moe_hash_balanced_table), else SplitMix64(hash_seed) output
 *                  number token_ids[s]+1, mod E.
 *           Ties go to the lower expert index.
 *   weights TOPK and HTOPK normalize=1: softmax over the k chosen logits (Eq. 1);
 *           TOPK and HTOPK normalize=0: softmax over all E logits at the chosen expert;
 *           KTOP1: softmax over the chosen expert's group; HASH: 1.
 * then assigns capacity slots in rank-major, token order: all first choices in
 * token order, then all second choices, and so on.  An expert's n-th
 * assignment (counting from 0) gets slot n if n < C, otherwise it is dropped.
 *
 * Inputs   x [S,d] and wg [d,E] (dtype), bias [E] fp32 or NULL: required when
 *          kind != HASH and logits_in == 0, else NULL.
 *          token_ids [S] int32 >= 0: required for HASH, else NULL (with a table, ids must be
 *          below hash_vocab; larger ids are out of contract and go to expert id mod E).
 *          noise [S,E] fp32 or NULL: only with temperature > 0.
 *          hash_table [hash_vocab] int32 in [0, E): HASH with hash_vocab > 0, else NULL.
 *          logits [S,E] fp32: input when logits_in == 1 (the raw logits; noise and
 *          temperature are applied to them).
 * Outputs  logits [S,E] fp32 (optional, NULL to skip; when logits_in == 0 the
 *          exact values the selection used, after noise and temperature), ids [S,k], weights [S,k] fp32,
 *          slots [S,k] (slot in the expert buffer, -1 = dropped), counts [E]
 *          (kept per expert, <= C), demand [E] (routed before the cap; NULL to
 *          skip), slot_src [E,C] (s*k + r of the assignment in each slot, -1 if
 *          empty).  Dropped assignments still report their id and weight.
 * Workspace device memory of at least moe_gate_workspace_size() bytes, 16-byte
 *          aligned; contents on entry are ignored.
 */
MOE_API moe_status moe_gate(const moe_gate_params* p, const void* x, const void* wg,
                    const float* bias, const int32_t* token_ids, const float* noise,
                    const int32_t* hash_table, float* logits, int32_t* ids, int32_t* slots,
                    float* weights, int32_t* counts, int32_t* demand, int32_t* slot_src,
                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Largest workspace moe_gate_noalloc serves from its fixed scratch (4 MiB). */
#define MOE_GATE_NOALLOC_MAX_BYTES (4u << 20)

/*
 * moe_gate_noalloc -- moe_gate for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, hosts that forbid
 * allocation): the same computation, arguments and outputs as moe_gate, without
 * the workspace arguments.  Its scratch is a fixed device array of
 * MOE_GATE_NOALLOC_MAX_BYTES inside the library, one per GPU, held from the
 * first call on that GPU until the process ends; the call itself allocates
 * nothing (no hipMalloc, no allocating library routine).
 *
 * Limit    the workspace moe_gate_workspace_size() reports for `p` must be at
 *          most MOE_GATE_NOALLOC_MAX_BYTES (the histogram, 4 * k * E * ceil(S/64)
 *          bytes, plus S * E * 4 bytes of logits for the Dense-To-Sparse and
 *          hierarchical gates that select in a kernel of their own); larger
 *          requests return MOE_ERR_UNSUPPORTED before any HIP call.
 * Scratch  every call on one GPU uses that GPU's one array: calls that overlap
 *          on one GPU (several streams or host threads at once) race and give
 *          undefined results.  Calls in order on one stream are safe; no
 *          contents carry over between calls (each call overwrites all the
 *          scratch it reads).
 * Errors   as moe_gate; the first call on a GPU may also return MOE_ERR_HIP if
 *          the scratch's device address cannot be looked up.
 */
MOE_API moe_status moe_gate_noalloc(const moe_gate_params* p, const void* x, const void* wg,
                            const float* bias, const int32_t* token_ids, const float* noise,
                            const int32_t* hash_table, float* logits, int32_t* ids, int32_t* slots,
                            float* weights, int32_t* counts, int32_t* demand, int32_t* slot_src,
                            hipStream_t stream);

/*
 * moe_hash_balanced_table -- the balanced assignment of the Hash Layer gate
 * (Sec. 3.1): token ids in order of decreasing frequency (ties: lower id) each
 * go to the expert with the smallest summed frequency so far (ties: lower
 * expert).  HOST memory: freq [vocab] (finite, >= 0), table [vocab] output in
 * [0, E).  Runs on the calling thread, no HIP call; pass the table to moe_gate
 * (copied to the device by the caller) with hash_vocab = vocab.
 */
MOE_API moe_status moe_hash_balanced_table(const double* freq, int32_t vocab, int32_t E, int32_t* table);

/* Parameters of moe_base_gate (host memory). */
typedef struct {
  int32_t S;          /* tokens; a multiple of E, with S / E <= 2048 */
  int32_t d;          /* model width (row length of x) */
  int32_t E;          /* experts */
  int32_t capacity;   /* C: slots per expert for the layout calls (S / E keeps every token) */
  int32_t logits_in;  /* 1 = `logits` is an input and x, wg, bias are NULL; 0 = projected */
  int32_t dtype;      /* moe_dtype of x and wg */
  int32_t max_rounds; /* auction rounds allowed per eps phase; 0 = 4096 */
} moe_base_params;

/* What the auction of moe_base_gate did (host memory). */
typedef struct {
  int32_t phases;     /* eps phases run */
  int32_t rounds;     /* bidding rounds, summed over phases */
  double eps;         /* eps of the last phase: the total score is within S * eps of the optimum */
} moe_base_info;

/* Bytes of device workspace moe_base_gate needs for `p`.  Fails with
 * MOE_ERR_INVALID_ARG for parameters moe_base_gate would reject. */
MOE_API moe_status moe_base_gate_workspace_size(const moe_base_params* p, size_t* bytes);

/*
 * moe_base_gate -- the BASE layer gate of Sec. 3.1: a balanced assignment in
 * which every expert receives exactly S / E tokens and the summed score
 * sum_s L[s, a_s] is as large as possible (a linear assignment problem), with
 * L[s,e] = sum_j x[s,j] * wg[j,e] + bias[e] the gate logits (fp32 accumulation)
 * as in moe_gate, or given.
 *
 * Solved by an auction with eps-scaling (Bertsekas): prices and bids in fp64,
 * eps from a quarter of the score range down to the range times 2^-30, so the
 * total is within S * info->eps of the optimum (exactly optimal when distinct
 * assignments' totals differ by more than that).  Equal bids go to the lower
 * token; results are bitwise reproducible.
 *
 * Outputs ids [S] (k = 1), weights [S] fp32 = sigmoid(L[s, ids[s]]) (the BASE
 * layer scales its expert's output by this), logits [S,E] fp32 (optional
 * output when logits_in == 0), and, as moe_gate with k = 1: slots [S], counts
 * [E], slot_src [E,C] in token order per expert.  prices [E] fp64 (device, may
 * be NULL): the auction's final expert prices p, a certificate of optimality:
 * with D = sum_s max_e (L[s,e] - p[e]) + (S/E) * sum_e p[e], an upper bound on
 * the optimum for any p, the returned total is at least D - S * info->eps, and
 * every token is within eps of its best L[s,e] - p[e].  info (host memory, may
 * be NULL) receives the auction's statistics.
 *
 * Unlike the other calls this one SYNCHRONIZES `stream`: the host enqueues the
 * auction's launches a few rounds ahead of the device, which reports its
 * progress and its end in a small pinned host buffer (one per host thread,
 * allocated on first use and kept until the process ends; without it, the
 * host enqueues batches of 64, then 128 rounds and reads the done flag after
 * each, as it also does when the environment sets HETUMOE_BASE_BATCHES=1); a
 * launch that finds the auction finished returns at once.
 * moe_base_gate_async below enqueues a fixed number of launches instead and
 * reads nothing back.  It returns
 * MOE_ERR_NOT_CONVERGED when a phase reaches max_rounds, and
 * MOE_ERR_INVALID_ARG when a score is infinite or NaN (found on the device
 * after the projection); outputs are then undefined.
 * Workspace device memory of at least moe_base_gate_workspace_size() bytes,
 *          16-byte aligned; contents on entry are ignored.
 */
MOE_API moe_status moe_base_gate(const moe_base_params* p, const void* x, const void* wg,
                                 const float* bias, float* logits, int32_t* ids, int32_t* slots,
                                 float* weights, int32_t* counts, int32_t* slot_src, double* prices,
                                 void* workspace, size_t workspace_bytes, moe_base_info* info,
                                 hipStream_t stream);

/* What the auction of moe_base_gate_async did (DEVICE memory, written by its
 * last kernel; 24 bytes, 8-byte aligned). */
typedef struct {
  int32_t phases;     /* eps phases run (0 when S == 0) */
  int32_t rounds;     /* bidding rounds, summed over phases */
  double eps;         /* eps of the last phase run */
  int32_t status;     /* 0 balanced assignment found; 1 not found within the rounds
                         enqueued or max_rounds; 2 a score is infinite or NaN */
  int32_t pad;
} moe_base_status;

/* Largest launch_rounds moe_base_gate_async accepts. */
#define MOE_BASE_MAX_LAUNCH_ROUNDS 16384

/*
 * moe_base_gate_async -- moe_base_gate without host synchronization, for
 * callers that capture their work in a HIP graph or cannot wait on the host.
 * The same kernels run with the same arguments and inputs, so when status->
 * status ends 0 every output is bitwise that of moe_base_gate, and the same
 * optimality bound holds with status->eps.
 *
 * Instead of reading the auction's done flag between batches, the call
 * enqueues exactly launch_rounds rounds (in [1, MOE_BASE_MAX_LAUNCH_ROUNDS];
 * one round is a bid, a resolve and a tail kernel, the tail kernel finishing
 * the rounds with few bidders in one workgroup; a round enqueued after the
 * auction has ended returns at once, in a few microseconds).  Rounds that
 * suffice are workload-dependent: moe_base_gate's info->rounds bounds them
 * from above (the workloads of 32768 tokens over 64 experts end within 64).  The
 * outcome is
 * written to `status` (device memory, required) by the call's last auction
 * kernel; no host read, memset or allocation is made.
 *
 * Outputs are always written and always in range: when status->status is 1
 * or 2, ids holds each token's expert as the unfinished auction left it (or
 * s mod E for a token holding none), so counts may exceed S / E and tokens
 * past the capacity get slot -1 as in moe_gate; weights may be NaN when
 * status->status is 2.  Argument errors are those of moe_base_gate, plus
 * MOE_ERR_INVALID_ARG for launch_rounds outside its range or a NULL or
 * misaligned status; no device-side failure is reported by the return value.
 * Workspace as for moe_base_gate; calls that overlap on one workspace race.
 */
MOE_API moe_status moe_base_gate_async(const moe_base_params* p, const void* x, const void* wg,
                                       const float* bias, float* logits, int32_t* ids, int32_t* slots,
                                       float* weights, int32_t* counts, int32_t* slot_src,
                                       double* prices, void* workspace, size_t workspace_bytes,
                                       int32_t launch_rounds, moe_base_status* status,
                                       hipStream_t stream);

/*
 * moe_dispatch -- step 2 of Algorithm 1 (Layout_Transform; Sec. 3.2, layout
 * transform): tokens routed to one expert become one contiguous buffer.
 *   xe[e,c,:] = x[slot_src[e,c] / k, :]   if slot_src[e,c] >= 0   (bit copy)
 *   xe[e,c,:] = 0                          otherwise
 * x [S,d]; ids, slots [S,k] and slot_src [E,C] as written by one moe_gate call
 * (the kernel walks tokens through ids/slots when k > 1, so that each row of x
 * is read once, and slots through slot_src when k = 1); xe [E,C,d] output.
 */
MOE_API moe_status moe_dispatch(const moe_layout* l, const void* x, const int32_t* ids,
                                const int32_t* slots, const int32_t* slot_src, void* xe,
                                hipStream_t stream);

/*
 * moe_combine -- step 6 of Algorithm 1 (Reverse_Layout_Transform) with the gate
 * weighting of step 4 / the second line of Eq. 1 applied here:
 *   y[s,:] = sum over r with slots[s,r] >= 0 of weights[s,r] * ye[ids[s,r], slots[s,r], :]
 * accumulated in fp32 in r order and rounded once; a token with no kept choice
 * gets a zero row.  ye [E,C,d], ids/slots/weights [S,k], y [S,d] output.
 */
MOE_API moe_status moe_combine(const moe_layout* l, const void* ye, const int32_t* ids,
                       const int32_t* slots, const float* weights, void* y,
                       hipStream_t stream);

/*
 * moe_dispatch_bwd -- gradient of moe_dispatch (adjoint of step 2):
 *   dx[s,:] = sum over r with slots[s,r] >= 0 of dxe[ids[s,r], slots[s,r], :]
 * accumulated in fp32 and rounded once.  dxe [E,C,d], dx [S,d] output.
 */
MOE_API moe_status moe_dispatch_bwd(const moe_layout* l, const void* dxe, const int32_t* ids,
                            const int32_t* slots, void* dx, hipStream_t stream);

/*
 * moe_combine_bwd -- gradient of moe_combine (adjoint of step 6):
 *   dye[e,c,:] = weights[s,r] * dy[s,:]   for (s,r) with s*k+r = slot_src[e,c] >= 0
 *   dye[e,c,:] = 0                         for empty slots
 *   dw[s,r]    = sum_j dy[s,j] * ye[e,c,j] for the slot (e,c) holding (s,r)
 *   dw[s,r]    = 0                          for dropped choices (slots[s,r] == -1)
 * dy [S,d]; ye [E,C,d] (NULL iff dw is NULL); ids, slots [S,k], slot_src [E,C]
 * and weights [S,k] as written by one moe_gate call; outputs dye [E,C,d] and
 * dw [S,k] fp32 or NULL.
 */
MOE_API moe_status moe_combine_bwd(const moe_layout* l, const void* dy, const void* ye,
                                   const int32_t* ids, const int32_t* slots,
                                   const int32_t* slot_src, const float* weights, void* dye,
                                   float* dw, hipStream_t stream);

/* Parameters of moe_gate_bwd (host memory). */
typedef struct {
  int32_t S, d, E, k;    /* as given to moe_gate */
  int32_t kind;          /* MOE_GATE_TOPK, MOE_GATE_KTOP1 or MOE_GATE_HTOPK (a hash gate has no gradient) */
  int32_t normalize;     /* as given to moe_gate */
  int32_t dtype;         /* moe_dtype of x, wg and dx */
  int32_t accumulate_dx; /* 1: dx += the gradient through the gate; 0: dx = that gradient */
  float aux_coef;        /* coefficient of the load-balancing loss, TOPK/HTOPK only; 0 = no loss */
  float temperature;     /* as given to moe_gate: > 0 means `logits` are (L + noise) / temperature
                            and the gradients are taken with respect to L; 0 = plain logits */
} moe_gate_bwd_params;

/* Bytes of device workspace moe_gate_bwd needs for `p`.  Fails with
 * MOE_ERR_INVALID_ARG for parameters moe_gate_bwd would reject. */
MOE_API moe_status moe_gate_bwd_workspace_size(const moe_gate_bwd_params* p, size_t* bytes);

/*
 * moe_gate_bwd -- gradient of step 1 of Algorithm 1 (the gate of Eq. 1), for
 * training the layer end to end (Sec. 2).  The loss reaches the gate through
 * the gate weights (dw, as written by moe_combine_bwd); the selection is held
 * fixed, since top-k and kTop1 are piecewise constant in the logits.
 *
 *   dL[s,e]  = sum_r dw[s,r] * d weights[s,r] / d L[s,e], with the weights of
 *              moe_gate recomputed from `logits`:
 *              TOPK normalize=1: dL[id_r] = w_r (dw_r - sum_r' w_r' dw_r'), 0 elsewhere;
 *              TOPK normalize=0: dL[e] = sum_r dw_r w_r ([e == id_r] - p_e), p = softmax(L[s,:]);
 *              KTOP1: for e in group g, dL[e] = dw_g w_g ([e == id_g] - p_g,e),
 *              p_g = softmax over the group.  HTOPK as TOPK.
 *            with temperature > 0, all of the above are taken with respect to the final
 *              (tempered) logits and then divided by the temperature.
 *            + with aux_coef != 0, the gradient of the load-balancing loss
 *              aux = aux_coef * E * sum_e f_e P_e, where f_e is the share of tokens
 *              whose first choice is e (held constant) and P_e the mean of p_e:
 *              aux_coef * E / S * p_e (f_e - sum_e' f_e' p_e').
 *   dwg[j,e] = sum_s x[s,j] dL[s,e]          (x^T dL; fp32)
 *   dbias[e] = sum_s dL[s,e]                 (fp32)
 *   dx[s,j]  = [dx[s,j] if accumulate_dx] + sum_e dL[s,e] wg[j,e], accumulated
 *              in fp32 and rounded once to dtype.
 * Sums over tokens run in a fixed order (no atomics): bitwise reproducible.
 *
 * Inputs   logits [S,E] fp32 (the logits moe_gate selected on, bias included),
 *          ids [S,k] (from the same moe_gate call), dw [S,k] fp32; x [S,d] when
 *          dwg != NULL; wg [d,E] when dx != NULL.  x and dx rows follow the
 *          alignment rule above; wg needs its natural alignment.
 * Outputs  each optional (NULL skips it): dlogits [S,E] fp32, dx [S,d] (read
 *          first when accumulate_dx), dwg [d,E] fp32, dbias [E] fp32, aux_loss
 *          [1] fp32 (the loss value; requires aux_coef != 0).
 * Workspace device memory of at least moe_gate_bwd_workspace_size() bytes,
 *          16-byte aligned; contents on entry are ignored.
 */
MOE_API moe_status moe_gate_bwd(const moe_gate_bwd_params* p, const void* x, const void* wg,
                                const float* logits, const int32_t* ids, const float* dw,
                                float* dlogits, void* dx, float* dwg, float* dbias,
                                float* aux_loss, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* Static description of a status code. */
MOE_API const char* moe_status_string(moe_status s);

/* Message for the last failed call on this host thread ("" if none). */
MOE_API const char* moe_last_error(void);

/* MOE_ABI_VERSION of the built library. */
MOE_API int32_t moe_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HETUMOE_H */
