// C ABI of the library: argument validation (before any HIP call), workspace
// sizing and kernel launches.  See include/hetumoe.h for the contract.
#include <stdarg.h>
#include <stddef.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <vector>

#include "hetumoe.h"
#include "common.hpp"
#include "kernels.hpp"

using namespace hetumoe;

// the asynchronous BASE call hands its caller's struct to the finish kernel
static_assert(sizeof(moe_base_status) == sizeof(BaseDevStatus) && sizeof(moe_base_status) == 24, "status layout");
static_assert(offsetof(moe_base_status, eps) == offsetof(BaseDevStatus, eps) &&
                  offsetof(moe_base_status, status) == offsetof(BaseDevStatus, status),
              "status layout");

namespace {

thread_local char g_last_error[512] = "";

moe_status fail(moe_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

moe_status ok() {
  g_last_error[0] = '\0';
  return MOE_OK;
}

moe_status hip_fail(hipError_t err, const char* what) {
  return fail(MOE_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(err), static_cast<int>(err));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t elt_size(int32_t dtype) { return dtype == MOE_BF16 ? 2 : 4; }

constexpr int64_t kI32Max = 2147483647;

int64_t hist_blocks(int64_t S) { return (S + kTokensPerHistBlock - 1) / kTokensPerHistBlock; }

// Checks shared by moe_gate and moe_gate_workspace_size.
moe_status check_gate_params(const moe_gate_params* p) {
  if (!p) return fail(MOE_ERR_INVALID_ARG, "params is NULL");
  if (p->dtype != MOE_F32 && p->dtype != MOE_BF16) return fail(MOE_ERR_INVALID_ARG, "dtype %d unknown", p->dtype);
  if (p->kind < MOE_GATE_TOPK || p->kind > MOE_GATE_HTOPK) return fail(MOE_ERR_INVALID_ARG, "gate kind %d unknown", p->kind);
  if (!std::isfinite(p->temperature) || p->temperature < 0.f)
    return fail(MOE_ERR_INVALID_ARG, "temperature must be finite and >= 0");
  if (p->hash_vocab < 0) return fail(MOE_ERR_INVALID_ARG, "hash_vocab = %d < 0", p->hash_vocab);
  if (p->kind != MOE_GATE_HASH && p->hash_vocab != 0) return fail(MOE_ERR_INVALID_ARG, "hash_vocab is for HASH only");
  if (p->kind != MOE_GATE_HTOPK && p->groups != 0) return fail(MOE_ERR_INVALID_ARG, "groups is for HTOPK only");
  if (p->S < 0) return fail(MOE_ERR_INVALID_ARG, "S = %d < 0", p->S);
  if (p->E < 1 || p->E > 1024) return fail(MOE_ERR_INVALID_ARG, "E = %d outside [1, 1024]", p->E);
  if (p->capacity < 0) return fail(MOE_ERR_INVALID_ARG, "capacity = %d < 0", p->capacity);
  if (static_cast<int64_t>(p->E) * p->capacity > kI32Max) return fail(MOE_ERR_INVALID_ARG, "E * capacity >= 2^31");
  if (p->normalize != 0 && p->normalize != 1) return fail(MOE_ERR_INVALID_ARG, "normalize must be 0 or 1");
  if (p->logits_in != 0 && p->logits_in != 1) return fail(MOE_ERR_INVALID_ARG, "logits_in must be 0 or 1");
  switch (p->kind) {
    case MOE_GATE_TOPK:
      if (p->k < 1 || p->k > 8 || p->k > p->E) return fail(MOE_ERR_INVALID_ARG, "TOPK needs 1 <= k <= min(E, 8), got k = %d, E = %d", p->k, p->E);
      break;
    case MOE_GATE_KTOP1:
      if (p->k < 1 || p->k > 8 || p->E % p->k != 0) return fail(MOE_ERR_INVALID_ARG, "KTOP1 needs 1 <= k <= 8 and E %% k == 0, got k = %d, E = %d", p->k, p->E);
      break;
    case MOE_GATE_HTOPK:
      if (p->groups < 1 || p->E % p->groups != 0)
        return fail(MOE_ERR_INVALID_ARG, "HTOPK needs groups >= 1 dividing E, got groups = %d, E = %d", p->groups, p->E);
      if (p->k < 1 || p->k > 8 || p->k > p->E / p->groups)
        return fail(MOE_ERR_INVALID_ARG, "HTOPK needs 1 <= k <= min(E / groups, 8), got k = %d", p->k);
      break;
    default:
      if (p->k != 1) return fail(MOE_ERR_INVALID_ARG, "HASH needs k = 1, got %d", p->k);
      if (p->logits_in) return fail(MOE_ERR_INVALID_ARG, "HASH takes no logits");
      if (p->temperature != 0.f) return fail(MOE_ERR_INVALID_ARG, "HASH takes no temperature");
      break;
  }
  if (static_cast<int64_t>(p->S) * p->k > kI32Max) return fail(MOE_ERR_INVALID_ARG, "S * k >= 2^31");
  const bool project = p->kind != MOE_GATE_HASH && !p->logits_in;
  if (project) {
    if (p->d < 1) return fail(MOE_ERR_INVALID_ARG, "d = %d < 1", p->d);
    if ((static_cast<int64_t>(p->d) * elt_size(p->dtype)) % 16 != 0)
      return fail(MOE_ERR_UNSUPPORTED, "row of x is %lld bytes; a multiple of 16 is required",
                  static_cast<long long>(p->d) * static_cast<long long>(elt_size(p->dtype)));
  }
  return MOE_OK;
}

// Gates whose selection runs on final logits in a kernel of its own: the
// hierarchical top-k, and any gate with a temperature (Dense-To-Sparse).
bool gate_extended(const moe_gate_params* p) {
  return p->kind != MOE_GATE_HASH && (p->kind == MOE_GATE_HTOPK || p->temperature > 0.f);
}

// Workspace: the histogram, int32 [k, E, ceil(S/64)]; for the extended gates
// also a logits buffer, fp32 [S, E], 256-byte aligned after the histogram.
size_t gate_hist_bytes(const moe_gate_params* p) {
  const size_t n = static_cast<size_t>(p->k) * static_cast<size_t>(hist_blocks(p->S)) * static_cast<size_t>(p->E);
  return n * sizeof(int32_t);
}

size_t gate_workspace_bytes(const moe_gate_params* p) {
  const size_t h = gate_hist_bytes(p);
  if (!gate_extended(p)) return h;
  return ((h + 255) & ~static_cast<size_t>(255)) + static_cast<size_t>(p->S) * static_cast<size_t>(p->E) * 4;
}

moe_status check_layout(const moe_layout* l, const char* who) {
  if (!l) return fail(MOE_ERR_INVALID_ARG, "%s: layout is NULL", who);
  if (l->dtype != MOE_F32 && l->dtype != MOE_BF16) return fail(MOE_ERR_INVALID_ARG, "%s: dtype %d unknown", who, l->dtype);
  if (l->S < 0 || l->d < 1 || l->E < 1 || l->E > 1024 || l->k < 1 || l->k > 8 || l->capacity < 0)
    return fail(MOE_ERR_INVALID_ARG, "%s: need S >= 0, d >= 1, 1 <= E <= 1024, 1 <= k <= 8, capacity >= 0 "
                "(got S=%d d=%d E=%d k=%d C=%d)", who, l->S, l->d, l->E, l->k, l->capacity);
  if (static_cast<int64_t>(l->S) * l->k > kI32Max || static_cast<int64_t>(l->E) * l->capacity > kI32Max)
    return fail(MOE_ERR_INVALID_ARG, "%s: S * k or E * capacity >= 2^31", who);
  if ((static_cast<int64_t>(l->d) * elt_size(l->dtype)) % 16 != 0)
    return fail(MOE_ERR_UNSUPPORTED, "%s: row is %lld bytes; a multiple of 16 is required", who,
                static_cast<long long>(l->d) * static_cast<long long>(elt_size(l->dtype)));
  return MOE_OK;
}

// A device buffer of n elements: required (non-NULL) when n > 0, with the
// given alignment.
moe_status need(const void* p, int64_t n, size_t align, const char* who, const char* name) {
  if (n > 0 && !p) return fail(MOE_ERR_INVALID_ARG, "%s: %s is NULL", who, name);
  if (p && !aligned(p, align))
    return fail(align == 16 ? MOE_ERR_UNSUPPORTED : MOE_ERR_INVALID_ARG, "%s: %s is not %zu-byte aligned", who, name, align);
  return MOE_OK;
}

// Checks shared by moe_gate_bwd and moe_gate_bwd_workspace_size.
moe_status check_gate_bwd_params(const moe_gate_bwd_params* p) {
  if (!p) return fail(MOE_ERR_INVALID_ARG, "params is NULL");
  if (p->dtype != MOE_F32 && p->dtype != MOE_BF16) return fail(MOE_ERR_INVALID_ARG, "dtype %d unknown", p->dtype);
  if (p->kind == MOE_GATE_HASH) return fail(MOE_ERR_INVALID_ARG, "a hash gate has no logits and no gradient");
  if (p->kind != MOE_GATE_TOPK && p->kind != MOE_GATE_KTOP1 && p->kind != MOE_GATE_HTOPK)
    return fail(MOE_ERR_INVALID_ARG, "gate kind %d unknown", p->kind);
  if (!std::isfinite(p->temperature) || p->temperature < 0.f)
    return fail(MOE_ERR_INVALID_ARG, "temperature must be finite and >= 0");
  if (p->S < 0) return fail(MOE_ERR_INVALID_ARG, "S = %d < 0", p->S);
  if (p->d < 1) return fail(MOE_ERR_INVALID_ARG, "d = %d < 1", p->d);
  if (p->E < 1 || p->E > 1024) return fail(MOE_ERR_INVALID_ARG, "E = %d outside [1, 1024]", p->E);
  if (p->normalize != 0 && p->normalize != 1) return fail(MOE_ERR_INVALID_ARG, "normalize must be 0 or 1");
  if (p->accumulate_dx != 0 && p->accumulate_dx != 1) return fail(MOE_ERR_INVALID_ARG, "accumulate_dx must be 0 or 1");
  if (p->kind != MOE_GATE_KTOP1 && (p->k < 1 || p->k > 8 || p->k > p->E))
    return fail(MOE_ERR_INVALID_ARG, "TOPK needs 1 <= k <= min(E, 8), got k = %d, E = %d", p->k, p->E);
  if (p->kind == MOE_GATE_KTOP1 && (p->k < 1 || p->k > 8 || p->E % p->k != 0))
    return fail(MOE_ERR_INVALID_ARG, "KTOP1 needs 1 <= k <= 8 and E %% k == 0, got k = %d, E = %d", p->k, p->E);
  if (static_cast<int64_t>(p->S) * p->k > kI32Max) return fail(MOE_ERR_INVALID_ARG, "S * k >= 2^31");
  if (!(p->aux_coef == p->aux_coef) || p->aux_coef > 3.0e38f || p->aux_coef < -3.0e38f)
    return fail(MOE_ERR_INVALID_ARG, "aux_coef must be finite");
  if (p->aux_coef != 0.f && p->kind == MOE_GATE_KTOP1)
    return fail(MOE_ERR_INVALID_ARG, "the load-balancing loss is defined for TOPK and HTOPK gates only");
  return MOE_OK;
}

// Workspace of moe_gate_bwd, each piece 256-byte aligned: dL [S,E] (used when
// the caller passes no dlogits), dL transposed [E, S rounded up to 64] as three
// bf16 planes (matrix cores only), first-choice counts [E] followed by per-4096-token counts, per
// wave block sums of the softmax and of dL [nb,E] each, softmax sums [E], and
// partial dW [nsplit,E,d] over token ranges.
struct GateBwdPlan {
  int nb, nsplit, split_tokens;
  bool mfma;
  int64_t s_pad;
  size_t off_dl, off_dlt, off_cnt, off_ppart, off_bpart, off_pe, off_wpart, total;
};

size_t align256(size_t n) { return (n + 255) & ~static_cast<size_t>(255); }

GateBwdPlan plan_gate_bwd(const moe_gate_bwd_params* p) {
  GateBwdPlan g{};
  const size_t S = static_cast<size_t>(p->S), E = static_cast<size_t>(p->E), d = static_cast<size_t>(p->d);
  g.nb = static_cast<int>(hist_blocks(p->S));
  g.mfma = gate_bwd_mfma_shape(p->dtype, p->E, p->d);
  g.s_pad = static_cast<int64_t>(g.nb) * kTokensPerHistBlock;
  // token ranges for dW: enough blocks to fill the chip (about 512 matrix-core
  // blocks of 256 columns, two per CU, or 1024 vector blocks of 64), each range
  // a whole number of 64-token blocks; matrix-core ranges keep at least 4 of
  // them where the batch allows, so that each block pipelines several chunks
  const int64_t per_split = g.mfma ? (p->d + 255) / 256 : ((p->d + 63) / 64) * ((p->E + 63) / 64);
  const int64_t target = g.mfma ? 512 : 1024;
  int64_t ns = (target + per_split - 1) / per_split;
  if (g.mfma && ns > g.nb / 4) ns = g.nb / 4;
  if (ns > g.nb) ns = g.nb;
  if (ns < 1) ns = 1;
  int64_t st = (static_cast<int64_t>(p->S) + ns - 1) / ns;
  st = (st + 63) / 64 * 64;
  if (st < 64) st = 64;
  g.split_tokens = static_cast<int>(st);
  g.nsplit = static_cast<int>((static_cast<int64_t>(p->S) + st - 1) / st);
  const size_t cblocks = (S + 4095) / 4096;
  size_t off = 0;
  g.off_dl = off;    off += align256(S * E * 4);
  g.off_dlt = off;   off += g.mfma ? align256(3 * static_cast<size_t>(g.s_pad) * E * 2) : 0;
  g.off_cnt = off;   off += align256((1 + cblocks) * E * 4);
  g.off_ppart = off; off += align256(static_cast<size_t>(g.nb) * E * 4);
  g.off_bpart = off; off += align256(static_cast<size_t>(g.nb) * E * 4);
  g.off_pe = off;    off += align256(E * 4);
  g.off_wpart = off; off += align256(static_cast<size_t>(g.nsplit) * E * d * 4);
  g.total = off;
  return g;
}

// Checks shared by moe_base_gate and moe_base_gate_workspace_size.
moe_status check_base_params(const moe_base_params* p) {
  if (!p) return fail(MOE_ERR_INVALID_ARG, "params is NULL");
  if (p->dtype != MOE_F32 && p->dtype != MOE_BF16) return fail(MOE_ERR_INVALID_ARG, "dtype %d unknown", p->dtype);
  if (p->S < 0) return fail(MOE_ERR_INVALID_ARG, "S = %d < 0", p->S);
  if (p->E < 1 || p->E > 1024) return fail(MOE_ERR_INVALID_ARG, "E = %d outside [1, 1024]", p->E);
  if (p->S % p->E != 0) return fail(MOE_ERR_INVALID_ARG, "BASE needs S %% E == 0, got S = %d, E = %d", p->S, p->E);
  if (p->S / p->E > kBaseMaxCap)
    return fail(MOE_ERR_UNSUPPORTED, "BASE needs S / E <= %d, got %d", kBaseMaxCap, p->S / p->E);
  if (p->capacity < 0) return fail(MOE_ERR_INVALID_ARG, "capacity = %d < 0", p->capacity);
  if (static_cast<int64_t>(p->E) * p->capacity > kI32Max) return fail(MOE_ERR_INVALID_ARG, "E * capacity >= 2^31");
  if (p->logits_in != 0 && p->logits_in != 1) return fail(MOE_ERR_INVALID_ARG, "logits_in must be 0 or 1");
  if (p->max_rounds < 0) return fail(MOE_ERR_INVALID_ARG, "max_rounds = %d < 0", p->max_rounds);
  if (!p->logits_in) {
    if (p->d < 1) return fail(MOE_ERR_INVALID_ARG, "d = %d < 1", p->d);
    if ((static_cast<int64_t>(p->d) * elt_size(p->dtype)) % 16 != 0)
      return fail(MOE_ERR_UNSUPPORTED, "row of x is %lld bytes; a multiple of 16 is required",
                  static_cast<long long>(p->d) * static_cast<long long>(elt_size(p->dtype)));
  }
  return MOE_OK;
}

// Workspace of moe_base_gate, each piece 256-byte aligned: hist int32 [E, nb];
// logits fp32 [S, E] (only when projected); price fp64 [E]; hold_v fp64 [S];
// hold_t, assign, bid_e int32 [S]; bid_v fp64 [S]; hold_n, bid_cnt int32 [E];
// counts int32 [2]; the auction state [2]; range partials fp32 [3, 256].
struct BasePlan {
  size_t off_hist, off_logits, off_price, off_hold_v, off_hold_t, off_hold_n, off_assign, off_bid_e, off_bid_v,
      off_bid_cnt, off_blist, off_counts, off_state, off_range, total;
};

BasePlan plan_base(const moe_base_params* p, bool own_logits) {
  BasePlan b{};
  const size_t S = static_cast<size_t>(p->S), E = static_cast<size_t>(p->E);
  size_t off = 0;
  b.off_hist = off;    off += align256(static_cast<size_t>(hist_blocks(p->S)) * E * 4);
  b.off_logits = off;  off += own_logits ? align256(S * E * 4) : 0;
  b.off_price = off;   off += align256(E * 8);
  b.off_hold_v = off;  off += align256(S * 8);
  b.off_hold_t = off;  off += align256(S * 4);
  b.off_hold_n = off;  off += align256(E * 4);
  b.off_assign = off;  off += align256(S * 4);
  b.off_bid_e = off;   off += align256(S * 4);
  b.off_bid_v = off;   off += align256(S * 8);
  b.off_bid_cnt = off; off += align256(E * 4);
  b.off_blist = off;   off += align256(S * 4);
  b.off_counts = off;  off += align256(4 * 4);
  b.off_state = off;   off += align256(2 * sizeof(BaseState));
  b.off_range = off;   off += align256(3 * kBaseRangeBlocks * sizeof(float));
  b.total = off;
  return b;
}

int nchunks(const moe_layout* l) {
  return static_cast<int>((static_cast<int64_t>(l->d) * elt_size(l->dtype)) / 16);
}

}  // namespace

#define CHECK(expr)                 \
  do {                              \
    moe_status _st = (expr);        \
    if (_st != MOE_OK) return _st;  \
  } while (0)

extern "C" {

int32_t moe_abi_version(void) { return MOE_ABI_VERSION; }

moe_status moe_gate_bwd_workspace_size(const moe_gate_bwd_params* p, size_t* bytes) {
  if (!bytes) return fail(MOE_ERR_INVALID_ARG, "bytes is NULL");
  CHECK(check_gate_bwd_params(p));
  *bytes = plan_gate_bwd(p).total;
  return ok();
}

moe_status moe_gate_bwd(const moe_gate_bwd_params* p, const void* x, const void* wg, const float* logits,
                        const int32_t* ids, const float* dw, float* dlogits, void* dx, float* dwg,
                        float* dbias, float* aux_loss, void* workspace, size_t workspace_bytes,
                        hipStream_t stream) {
  static const char* who = "moe_gate_bwd";
  CHECK(check_gate_bwd_params(p));
  const int64_t S = p->S, E = p->E, k = p->k, d = p->d;
  const size_t elt = elt_size(p->dtype);
  CHECK(need(logits, S * E, 4, who, "logits"));
  CHECK(need(ids, S * k, 4, who, "ids"));
  CHECK(need(dw, S * k, 4, who, "dw"));
  CHECK(need(dlogits, 0, 4, who, "dlogits"));
  CHECK(need(dbias, 0, 4, who, "dbias"));
  CHECK(need(aux_loss, 0, 4, who, "aux_loss"));
  if (aux_loss && p->aux_coef == 0.f) return fail(MOE_ERR_INVALID_ARG, "%s: aux_loss needs aux_coef != 0", who);
  if (dwg || dx) {
    if ((d * static_cast<int64_t>(elt)) % 16 != 0)
      return fail(MOE_ERR_UNSUPPORTED, "%s: row of x / dx is %lld bytes; a multiple of 16 is required", who,
                  static_cast<long long>(d * static_cast<int64_t>(elt)));
  }
  if (dwg) {
    CHECK(need(dwg, d * E, 4, who, "dwg"));
    CHECK(need(x, S * d, 16, who, "x"));
  }
  if (dx) {
    CHECK(need(dx, S * d, 16, who, "dx"));
    CHECK(need(wg, d * E, elt, who, "wg"));
  }
  const GateBwdPlan g = plan_gate_bwd(p);
  if (workspace_bytes < g.total) return fail(MOE_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", who, workspace_bytes, g.total);
  if (g.total > 0 && !workspace) return fail(MOE_ERR_WORKSPACE, "%s: workspace is NULL", who);
  if (workspace && !aligned(workspace, 16)) return fail(MOE_ERR_WORKSPACE, "%s: workspace is not 16-byte aligned", who);

  char* ws = static_cast<char*>(workspace);
  GateBwdArgs a{};
  a.S = p->S; a.d = p->d; a.E = p->E; a.k = p->k; a.nb = g.nb;
  a.kind = p->kind; a.normalize = p->normalize; a.dtype = p->dtype; a.accumulate = p->accumulate_dx;
  a.aux_coef = p->aux_coef; a.temperature = p->temperature; a.nsplit = g.nsplit; a.split_tokens = g.split_tokens;
  a.mfma_dw = (g.mfma && dwg) ? 1 : 0;
  // the matrix-core dx reads W rows and dL with 16-byte loads
  a.mfma_dx = (g.mfma && dx && aligned(wg, 16) && (!dlogits || aligned(dlogits, 16))) ? 1 : 0;
  a.s_pad = g.s_pad;
  // with dW wanted, its reduction launch also takes db and the balance loss
  a.sums_in_reduce = (dwg && p->E <= 64) ? 1 : 0;
  a.x = x; a.wg = wg; a.logits = logits; a.ids = ids; a.dw = dw;
  a.dl = dlogits ? dlogits : reinterpret_cast<float*>(ws + g.off_dl);
  a.dlt = a.mfma_dw ? reinterpret_cast<uint16_t*>(ws + g.off_dlt) : nullptr;
  a.dx = dx; a.dwg = dwg; a.dbias = dbias; a.aux_loss = aux_loss;
  a.cnt = reinterpret_cast<int32_t*>(ws + g.off_cnt);
  a.ppart = reinterpret_cast<float*>(ws + g.off_ppart);
  a.bpart = reinterpret_cast<float*>(ws + g.off_bpart);
  a.pe = reinterpret_cast<float*>(ws + g.off_pe);
  a.wpart = reinterpret_cast<float*>(ws + g.off_wpart);
  hipError_t err = launch_gate_bwd_dl(a, stream);
  if (err != hipSuccess) return hip_fail(err, "moe_gate_bwd: dL kernel launch");
  if (dwg) {
    err = launch_gate_bwd_dwg(a, stream);
    if (err != hipSuccess) return hip_fail(err, "moe_gate_bwd: dW kernel launch");
  }
  if (dx) {
    err = launch_gate_bwd_dx(a, stream);
    if (err != hipSuccess) return hip_fail(err, "moe_gate_bwd: dx kernel launch");
  }
  return ok();
}

const char* moe_status_string(moe_status s) {
  switch (s) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG";
    case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
    case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE";
    case MOE_ERR_HIP: return "MOE_ERR_HIP";
    case MOE_ERR_NOT_CONVERGED: return "MOE_ERR_NOT_CONVERGED";
  }
  return "unknown moe_status";
}

const char* moe_last_error(void) { return g_last_error; }

moe_status moe_gate_workspace_size(const moe_gate_params* p, size_t* bytes) {
  if (!bytes) return fail(MOE_ERR_INVALID_ARG, "bytes is NULL");
  CHECK(check_gate_params(p));
  *bytes = gate_workspace_bytes(p);
  return ok();
}

}  // extern "C"

namespace {

// Scratch of moe_gate_noalloc: the gate's workspace in device memory the library
// owns, one copy per GPU, held until the process ends.  Host code uses only the
// address hipGetSymbolAddress returns for the current device, never the name.
constexpr size_t kGateScratchBytes = MOE_GATE_NOALLOC_MAX_BYTES;
__device__ __align__(256) unsigned char scratch[kGateScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch (looked up once per device;
// every thread that looks it up stores the same address).
moe_status scratch_address(const char* who, void** out) {
  int dev = -1;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return hip_fail(err, "moe_gate_noalloc: hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(MOE_ERR_UNSUPPORTED, "%s: device %d beyond the %d served", who, dev, kMaxDevices);
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return hip_fail(err, "moe_gate_noalloc: hipGetSymbolAddress(scratch)");
    if (!p) return fail(MOE_ERR_HIP, "%s: hipGetSymbolAddress(scratch) gave NULL", who);
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return MOE_OK;
}

// moe_gate and moe_gate_noalloc: with `noalloc` the workspace arguments are
// ignored and the gate runs in the library's scratch.
moe_status gate_call(const char* who, bool noalloc, const moe_gate_params* p, const void* x, const void* wg,
                     const float* bias, const int32_t* token_ids, const float* noise, const int32_t* hash_table,
                     float* logits, int32_t* ids, int32_t* slots, float* weights, int32_t* counts, int32_t* demand,
                     int32_t* slot_src, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  CHECK(check_gate_params(p));
  const int64_t S = p->S, E = p->E, k = p->k, C = p->capacity;
  const size_t elt = elt_size(p->dtype);
  if (p->kind == MOE_GATE_HASH) {
    CHECK(need(token_ids, S, 4, who, "token_ids"));
    if (x || wg || bias || logits || noise) return fail(MOE_ERR_INVALID_ARG, "%s: HASH takes no x, wg, bias, logits or noise", who);
    if (p->hash_vocab > 0) CHECK(need(hash_table, p->hash_vocab, 4, who, "hash_table"));
    else if (hash_table) return fail(MOE_ERR_INVALID_ARG, "%s: hash_table needs hash_vocab > 0", who);
  } else {
    if (hash_table) return fail(MOE_ERR_INVALID_ARG, "%s: hash_table is only for HASH", who);
    if (noise && p->temperature == 0.f) return fail(MOE_ERR_INVALID_ARG, "%s: noise needs a temperature > 0", who);
    CHECK(need(noise, 0, 4, who, "noise"));
    if (p->logits_in) {
      CHECK(need(logits, S * E, 4, who, "logits"));
      if (x || wg || bias || token_ids) return fail(MOE_ERR_INVALID_ARG, "%s: with logits_in, x, wg, bias and token_ids must be NULL", who);
    } else {
      CHECK(need(x, S * p->d, 16, who, "x"));
      CHECK(need(wg, static_cast<int64_t>(p->d) * E, elt, who, "wg"));
      CHECK(need(bias, 0, 4, who, "bias"));
      CHECK(need(logits, 0, 4, who, "logits"));
      if (token_ids) return fail(MOE_ERR_INVALID_ARG, "%s: token_ids is only for HASH", who);
    }
  }
  CHECK(need(ids, S * k, 4, who, "ids"));
  CHECK(need(slots, S * k, 4, who, "slots"));
  CHECK(need(weights, S * k, 4, who, "weights"));
  CHECK(need(counts, E, 4, who, "counts"));
  CHECK(need(demand, 0, 4, who, "demand"));
  CHECK(need(slot_src, E * C, 4, who, "slot_src"));
  const size_t ws = gate_workspace_bytes(p);
  if (noalloc) {
    if (ws > kGateScratchBytes)
      return fail(MOE_ERR_UNSUPPORTED, "%s: this gate needs %zu bytes of scratch; the fixed scratch holds %zu "
                  "(use moe_gate with a workspace)", who, ws, kGateScratchBytes);
    CHECK(scratch_address(who, &workspace));
    workspace_bytes = kGateScratchBytes;
  } else {
    if (workspace_bytes < ws) return fail(MOE_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", who, workspace_bytes, ws);
    if (ws > 0 && !workspace) return fail(MOE_ERR_WORKSPACE, "%s: workspace is NULL", who);
    if (workspace && !aligned(workspace, 16)) return fail(MOE_ERR_WORKSPACE, "%s: workspace is not 16-byte aligned", who);
  }

  const int nb = static_cast<int>(hist_blocks(S));
  int32_t* hist = static_cast<int32_t*>(workspace);
  hipError_t err;

  RouteArgs fused{};
  fused.S = p->S; fused.d = p->d; fused.E = p->E; fused.k = p->k; fused.nb = nb;
  fused.kind = p->kind; fused.normalize = p->normalize; fused.logits_in = 0; fused.dtype = p->dtype;
  fused.x = x; fused.wg = wg; fused.bias = bias; fused.logits = logits;
  fused.ids = ids; fused.weights = weights; fused.hist = hist;
  fused.groups = p->groups; fused.temperature = p->temperature; fused.noise = noise;
  if (gate_extended(p) && !p->logits_in && route_fuses_extended(fused)) {
    // projection, noise, temperature and selection in one kernel: the final
    // logits never leave it unless the caller asks for them
    err = launch_route(fused, stream);
    if (err != hipSuccess) return hip_fail(err, "moe_gate: route kernel launch");
  } else if (gate_extended(p)) {
    // raw logits (projected into the workspace, or given), then noise,
    // temperature and selection in a kernel of their own
    float* wsl = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                          ((gate_hist_bytes(p) + 255) & ~static_cast<size_t>(255)));
    const float* raw = logits;
    float* fin = wsl;
    if (!p->logits_in) {
      // projection only: a one-choice top-k pass writes the logits; its ids,
      // weights and histogram are overwritten below
      RouteArgs ra{};
      ra.S = p->S; ra.d = p->d; ra.E = p->E; ra.k = 1; ra.nb = nb;
      ra.kind = MOE_GATE_TOPK; ra.normalize = 0; ra.logits_in = 0; ra.dtype = p->dtype;
      ra.x = x; ra.wg = wg; ra.bias = bias; ra.logits = wsl;
      ra.ids = ids; ra.weights = weights; ra.hist = hist;
      err = launch_route(ra, stream);
      if (err != hipSuccess) return hip_fail(err, "moe_gate: route kernel launch");
      raw = wsl;
      fin = logits ? logits : wsl;
    }
    SelectArgs sel{};
    sel.S = p->S; sel.E = p->E; sel.k = p->k; sel.nb = nb; sel.kind = p->kind; sel.normalize = p->normalize;
    sel.groups = p->groups; sel.temperature = p->temperature;
    sel.raw = raw; sel.noise = noise; sel.fin = fin; sel.ids = ids; sel.weights = weights; sel.hist = hist;
    err = launch_select_ext(sel, stream);
    if (err != hipSuccess) return hip_fail(err, "moe_gate: selection kernel launch");
  } else {
    RouteArgs ra{};
    ra.S = p->S; ra.d = p->d; ra.E = p->E; ra.k = p->k; ra.nb = nb;
    ra.kind = p->kind; ra.normalize = p->normalize; ra.logits_in = p->logits_in; ra.dtype = p->dtype;
    ra.hash_seed = p->hash_seed;
    ra.x = x; ra.wg = wg; ra.bias = bias; ra.token_ids = token_ids; ra.logits = logits;
    ra.hash_table = hash_table; ra.hash_vocab = p->hash_vocab;
    ra.ids = ids; ra.weights = weights; ra.hist = hist;
    err = launch_route(ra, stream);
    if (err != hipSuccess) return hip_fail(err, "moe_gate: route kernel launch");
  }

  ScanArgs sa{};
  sa.E = p->E; sa.k = p->k; sa.nb = nb; sa.C = p->capacity;
  sa.hist = hist; sa.counts = counts; sa.demand = demand; sa.slot_src = slot_src;
  AssignArgs aa{};
  aa.S = p->S; aa.E = p->E; aa.k = p->k; aa.nb = nb; aa.C = p->capacity;
  aa.ids = ids; aa.offs = hist; aa.slots = slots; aa.slot_src = slot_src;
  err = launch_scan_assign(sa, aa, stream);
  if (err != hipSuccess) return hip_fail(err, "moe_gate: scan / assign kernel launch");
  return ok();
}

}  // namespace

extern "C" {

moe_status moe_gate(const moe_gate_params* p, const void* x, const void* wg, const float* bias,
                    const int32_t* token_ids, const float* noise, const int32_t* hash_table, float* logits,
                    int32_t* ids, int32_t* slots, float* weights, int32_t* counts, int32_t* demand,
                    int32_t* slot_src, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return gate_call("moe_gate", false, p, x, wg, bias, token_ids, noise, hash_table, logits, ids, slots, weights,
                   counts, demand, slot_src, workspace, workspace_bytes, stream);
}

moe_status moe_gate_noalloc(const moe_gate_params* p, const void* x, const void* wg, const float* bias,
                            const int32_t* token_ids, const float* noise, const int32_t* hash_table, float* logits,
                            int32_t* ids, int32_t* slots, float* weights, int32_t* counts, int32_t* demand,
                            int32_t* slot_src, hipStream_t stream) {
  return gate_call("moe_gate_noalloc", true, p, x, wg, bias, token_ids, noise, hash_table, logits, ids, slots,
                   weights, counts, demand, slot_src, nullptr, 0, stream);
}

moe_status moe_hash_balanced_table(const double* freq, int32_t vocab, int32_t E, int32_t* table) {
  if (!freq || !table) return fail(MOE_ERR_INVALID_ARG, "moe_hash_balanced_table: freq and table are required");
  if (vocab < 1) return fail(MOE_ERR_INVALID_ARG, "moe_hash_balanced_table: vocab = %d < 1", vocab);
  if (E < 1 || E > 1024) return fail(MOE_ERR_INVALID_ARG, "moe_hash_balanced_table: E = %d outside [1, 1024]", E);
  for (int32_t t = 0; t < vocab; ++t)
    if (!std::isfinite(freq[t]) || freq[t] < 0.0)
      return fail(MOE_ERR_INVALID_ARG, "moe_hash_balanced_table: freq[%d] is not a finite value >= 0", t);
  std::vector<int32_t> order(static_cast<size_t>(vocab));
  for (int32_t t = 0; t < vocab; ++t) order[t] = t;
  // decreasing frequency; the stable sort keeps equal frequencies in id order
  std::stable_sort(order.begin(), order.end(), [freq](int32_t a, int32_t b) { return freq[a] > freq[b]; });
  std::vector<double> load(static_cast<size_t>(E), 0.0);
  for (int32_t t : order) {
    int32_t best = 0;
    for (int32_t e = 1; e < E; ++e)
      if (load[e] < load[best]) best = e;  // strict: ties keep the lower expert
    table[t] = best;
    load[best] += freq[t];
  }
  return ok();
}

moe_status moe_dispatch(const moe_layout* l, const void* x, const int32_t* ids, const int32_t* slots,
                        const int32_t* slot_src, void* xe, hipStream_t stream) {
  static const char* who = "moe_dispatch";
  CHECK(check_layout(l, who));
  const int64_t rows = static_cast<int64_t>(l->E) * l->capacity;
  const int64_t Sk = static_cast<int64_t>(l->S) * l->k;
  CHECK(need(x, static_cast<int64_t>(l->S) * l->d, 16, who, "x"));
  CHECK(need(ids, Sk, 4, who, "ids"));
  CHECK(need(slots, Sk, 4, who, "slots"));
  CHECK(need(slot_src, rows, 4, who, "slot_src"));
  CHECK(need(xe, rows * l->d, 16, who, "xe"));
  RowArgs a{};
  a.rows = rows; a.nch = nchunks(l); a.S = l->S; a.E = l->E; a.k = l->k; a.C = l->capacity; a.dtype = l->dtype;
  a.src = x; a.ids = ids; a.slots = slots; a.slot_src = slot_src; a.dst = xe;
  const hipError_t err = launch_dispatch(a, stream);
  if (err != hipSuccess) return hip_fail(err, "moe_dispatch: kernel launch");
  return ok();
}

static moe_status combine_common(const char* who, const moe_layout* l, const void* src,
                                 const int32_t* ids, const int32_t* slots, const float* weights,
                                 void* out, bool weighted, hipStream_t stream) {
  CHECK(check_layout(l, who));
  const int64_t S = l->S, k = l->k;
  CHECK(need(src, static_cast<int64_t>(l->E) * l->capacity * l->d, 16, who, weighted ? "ye" : "dxe"));
  CHECK(need(ids, S * k, 4, who, "ids"));
  CHECK(need(slots, S * k, 4, who, "slots"));
  if (weighted) CHECK(need(weights, S * k, 4, who, "weights"));
  CHECK(need(out, S * l->d, 16, who, weighted ? "y" : "dx"));
  RowArgs a{};
  a.rows = S; a.nch = nchunks(l); a.S = l->S; a.E = l->E; a.k = l->k; a.C = l->capacity; a.dtype = l->dtype;
  a.src = src; a.ids = ids; a.slots = slots; a.weights = weights; a.dst = out;
  const hipError_t err = launch_combine(a, weighted, stream);
  if (err != hipSuccess) return hip_fail(err, weighted ? "moe_combine: kernel launch" : "moe_dispatch_bwd: kernel launch");
  return ok();
}

moe_status moe_combine(const moe_layout* l, const void* ye, const int32_t* ids, const int32_t* slots,
                       const float* weights, void* y, hipStream_t stream) {
  return combine_common("moe_combine", l, ye, ids, slots, weights, y, true, stream);
}

moe_status moe_dispatch_bwd(const moe_layout* l, const void* dxe, const int32_t* ids,
                            const int32_t* slots, void* dx, hipStream_t stream) {
  return combine_common("moe_dispatch_bwd", l, dxe, ids, slots, nullptr, dx, false, stream);
}

moe_status moe_combine_bwd(const moe_layout* l, const void* dy, const void* ye, const int32_t* ids,
                           const int32_t* slots, const int32_t* slot_src, const float* weights, void* dye,
                           float* dw, hipStream_t stream) {
  static const char* who = "moe_combine_bwd";
  CHECK(check_layout(l, who));
  const int64_t S = l->S, k = l->k;
  const int64_t rows = static_cast<int64_t>(l->E) * l->capacity;
  CHECK(need(dy, S * l->d, 16, who, "dy"));
  CHECK(need(ids, S * k, 4, who, "ids"));
  CHECK(need(slots, S * k, 4, who, "slots"));
  CHECK(need(slot_src, rows, 4, who, "slot_src"));
  CHECK(need(weights, S * k, 4, who, "weights"));
  CHECK(need(dye, rows * l->d, 16, who, "dye"));
  if (dw) {
    CHECK(need(ye, rows * l->d, 16, who, "ye"));
    CHECK(need(dw, S * k, 4, who, "dw"));
  } else if (ye) {
    return fail(MOE_ERR_INVALID_ARG, "%s: ye must be NULL when dw is NULL", who);
  }
  RowArgs a{};
  a.rows = rows; a.nch = nchunks(l); a.S = l->S; a.E = l->E; a.k = l->k; a.C = l->capacity; a.dtype = l->dtype;
  a.src = dy; a.aux = ye; a.ids = ids; a.slots = slots; a.slot_src = slot_src; a.weights = weights; a.dst = dye;
  a.dw = dw;
  const hipError_t err = launch_combine_bwd(a, stream);
  if (err != hipSuccess) return hip_fail(err, "moe_combine_bwd: kernel launch");
  return ok();
}

moe_status moe_base_gate_workspace_size(const moe_base_params* p, size_t* bytes) {
  if (!bytes) return fail(MOE_ERR_INVALID_ARG, "bytes is NULL");
  CHECK(check_base_params(p));
  *bytes = plan_base(p, !p->logits_in).total;
  return ok();
}

}  // extern "C"

namespace {

// moe_base_gate and moe_base_gate_async: with launch_rounds == 0 the host reads
// the auction's state between batches of rounds (synchronous, info filled);
// otherwise exactly launch_rounds rounds are enqueued, nothing is read back,
// and the outcome goes to the device struct dstatus.
moe_status base_gate_run(const char* who, const moe_base_params* p, const void* x, const void* wg, const float* bias,
                         float* logits, int32_t* ids, int32_t* slots, float* weights, int32_t* counts,
                         int32_t* slot_src, double* prices, void* workspace, size_t workspace_bytes,
                         moe_base_info* info, int launch_rounds, moe_base_status* dstatus, hipStream_t stream) {
  CHECK(check_base_params(p));
  const int64_t S = p->S, E = p->E, C = p->capacity;
  const size_t elt = elt_size(p->dtype);
  if (p->logits_in) {
    CHECK(need(logits, S * E, 4, who, "logits"));
    if (x || wg || bias) return fail(MOE_ERR_INVALID_ARG, "%s: with logits_in, x, wg and bias must be NULL", who);
  } else {
    CHECK(need(x, S * p->d, 16, who, "x"));
    CHECK(need(wg, static_cast<int64_t>(p->d) * E, elt, who, "wg"));
    CHECK(need(bias, 0, 4, who, "bias"));
    CHECK(need(logits, 0, 4, who, "logits"));
  }
  CHECK(need(ids, S, 4, who, "ids"));
  CHECK(need(slots, S, 4, who, "slots"));
  CHECK(need(weights, S, 4, who, "weights"));
  CHECK(need(counts, E, 4, who, "counts"));
  CHECK(need(slot_src, E * C, 4, who, "slot_src"));
  CHECK(need(prices, 0, 8, who, "prices"));
  // the workspace size does not depend on whether the logits are returned
  const BasePlan b = plan_base(p, !p->logits_in);
  if (workspace_bytes < b.total) return fail(MOE_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", who, workspace_bytes, b.total);
  if (!workspace) return fail(MOE_ERR_WORKSPACE, "%s: workspace is NULL", who);
  if (!aligned(workspace, 16)) return fail(MOE_ERR_WORKSPACE, "%s: workspace is not 16-byte aligned", who);
  if (info) *info = moe_base_info{0, 0, 0.0};

  char* ws = static_cast<char*>(workspace);
  const int nb = static_cast<int>(hist_blocks(S));
  int32_t* hist = reinterpret_cast<int32_t*>(ws + b.off_hist);
  hipError_t err;
  const float* L = logits;
  if (!p->logits_in) {
    float* out = logits ? logits : reinterpret_cast<float*>(ws + b.off_logits);
    // projection only: a one-choice top-k pass writes the logits; its ids,
    // weights and histogram are overwritten by the auction's outputs
    RouteArgs ra{};
    ra.S = p->S; ra.d = p->d; ra.E = p->E; ra.k = 1; ra.nb = nb;
    ra.kind = MOE_GATE_TOPK; ra.normalize = 0; ra.logits_in = 0; ra.dtype = p->dtype;
    ra.x = x; ra.wg = wg; ra.bias = bias; ra.logits = out;
    ra.ids = ids; ra.weights = weights; ra.hist = hist;
    if (p->S > 0) {
      err = launch_route(ra, stream);
      if (err != hipSuccess) return hip_fail(err, "moe_base_gate: route kernel launch");
    }
    L = out;
  }
  BaseArgs a{};
  a.S = p->S; a.E = p->E; a.cap = p->S / p->E; a.nb = nb;
  a.max_rounds = p->max_rounds > 0 ? p->max_rounds : 4096;
  a.logits = L;
  a.price = reinterpret_cast<double*>(ws + b.off_price);
  a.hold_v = reinterpret_cast<double*>(ws + b.off_hold_v);
  a.hold_t = reinterpret_cast<int32_t*>(ws + b.off_hold_t);
  a.hold_n = reinterpret_cast<int32_t*>(ws + b.off_hold_n);
  a.assign = reinterpret_cast<int32_t*>(ws + b.off_assign);
  a.bid_e = reinterpret_cast<int32_t*>(ws + b.off_bid_e);
  a.bid_v = reinterpret_cast<double*>(ws + b.off_bid_v);
  a.bid_cnt = reinterpret_cast<int32_t*>(ws + b.off_bid_cnt);
  a.blist = reinterpret_cast<int32_t*>(ws + b.off_blist);
  a.counts = reinterpret_cast<int32_t*>(ws + b.off_counts);
  a.state = reinterpret_cast<BaseState*>(ws + b.off_state);
  a.range_part = reinterpret_cast<float*>(ws + b.off_range);
  a.ids = ids; a.weights = weights; a.hist = hist; a.prices_out = prices;
  if (launch_rounds > 0) {
    err = run_base_auction_async(a, launch_rounds, reinterpret_cast<BaseDevStatus*>(dstatus), stream);
    if (err != hipSuccess) return hip_fail(err, "moe_base_gate_async: auction launch");
  } else {
    BaseStats stats{};
    err = run_base_auction(a, stream, &stats);
    if (err != hipSuccess) return hip_fail(err, "moe_base_gate: auction");
    if (info) *info = moe_base_info{stats.phases, stats.rounds, stats.eps};
    if (stats.bad_scores) return fail(MOE_ERR_INVALID_ARG, "%s: a score is infinite or NaN", who);
    if (stats.not_converged)
      return fail(MOE_ERR_NOT_CONVERGED, "%s: no balanced assignment after %d rounds of a phase", who, a.max_rounds);
  }

  ScanArgs sa{};
  sa.E = p->E; sa.k = 1; sa.nb = nb; sa.C = p->capacity;
  sa.hist = hist; sa.counts = counts; sa.demand = nullptr; sa.slot_src = slot_src;
  AssignArgs aa{};
  aa.S = p->S; aa.E = p->E; aa.k = 1; aa.nb = nb; aa.C = p->capacity;
  aa.ids = ids; aa.offs = hist; aa.slots = slots; aa.slot_src = slot_src;
  err = launch_scan_assign(sa, aa, stream);
  if (err != hipSuccess) return hip_fail(err, "moe_base_gate: scan / assign kernel launch");
  return ok();
}


}  // namespace

extern "C" {

moe_status moe_base_gate(const moe_base_params* p, const void* x, const void* wg, const float* bias, float* logits,
                         int32_t* ids, int32_t* slots, float* weights, int32_t* counts, int32_t* slot_src,
                         double* prices, void* workspace, size_t workspace_bytes, moe_base_info* info,
                         hipStream_t stream) {
  return base_gate_run("moe_base_gate", p, x, wg, bias, logits, ids, slots, weights, counts, slot_src, prices,
                       workspace, workspace_bytes, info, 0, nullptr, stream);
}

moe_status moe_base_gate_async(const moe_base_params* p, const void* x, const void* wg, const float* bias,
                               float* logits, int32_t* ids, int32_t* slots, float* weights, int32_t* counts,
                               int32_t* slot_src, double* prices, void* workspace, size_t workspace_bytes,
                               int32_t launch_rounds, moe_base_status* status, hipStream_t stream) {
  static const char* who = "moe_base_gate_async";
  if (launch_rounds < 1 || launch_rounds > MOE_BASE_MAX_LAUNCH_ROUNDS)
    return fail(MOE_ERR_INVALID_ARG, "%s: launch_rounds = %d outside [1, %d]", who, launch_rounds,
                MOE_BASE_MAX_LAUNCH_ROUNDS);
  if (!status) return fail(MOE_ERR_INVALID_ARG, "%s: status is NULL", who);
  if (!aligned(status, 8)) return fail(MOE_ERR_INVALID_ARG, "%s: status is not 8-byte aligned", who);
  return base_gate_run(who, p, x, wg, bias, logits, ids, slots, weights, counts, slot_src, prices, workspace,
                       workspace_bytes, nullptr, launch_rounds, status, stream);
}

}  // extern "C"
