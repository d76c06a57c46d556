// ea_api.hip -- the C ABI: argument checks, buffer sizes and the launch
// sequence of the forward (tau solver with the mask's row tables -> sparse
// forward with the column tables) and backward (delta -> dK/dV -> dQ) passes.
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "../../include/entmax_attn.h"
#include "ea_internal.h"

// Scratch of entmax_attn_bwd_noalloc: delta (one fp32 per row) lives here
// instead of in a caller workspace.  Each device holds its own copy for the
// life of the process.  In host code `scratch` only names the symbol: its
// device address comes from hipGetSymbolAddress (scratch_for below), taken
// once per device with that device current, and only that address is passed
// to kernels.
static __device__ __align__(256) float scratch[EA_NOALLOC_MAX_ROWS];

namespace ea {

int gamma_kind(float alpha) {
  if (alpha == 2.0f) return 1;
  if (alpha == 1.5f) return 2;
  if (alpha == 1.25f) return 4;
  return 0;
}

namespace {

constexpr int DEFAULT_MAX_ITER = 12;
constexpr float DEFAULT_TOL = 1e-5f;
constexpr int MAX_ITER_CAP = 64;
// Candidate-cache entries per list (see entmax_attn_sizes); a slot holds
// two lists per row of a workgroup.
constexpr int TAU_CACHE_CAP = 192;
static_assert(TAU_CACHE_CAP % 16 == 0, "the solver reads lists in batches of 16 entries");
constexpr int SOLVE_QUAD_CAP = 96;
static_assert(SOLVE_QUAD_CAP % 8 == 0, "the solver reads lists in batches of 8 quads");
constexpr size_t SOLVE_SLOT_BYTES = solve_slot_bytes(SOLVE_QUAD_CAP);
static_assert(SOLVE_SLOT_BYTES % (2 * SOLVE_THREADS * sizeof(CandEntry) * 8) == 0,
              "a refilled slot holds a multiple of 8 single entries per list");
constexpr size_t TAU_SLOT_BYTES = (size_t)TAU_CACHE_CAP * 2 * TAU_ROWS * sizeof(CandEntry);

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct Dims {
  int64_t BH, n, d, T, elems;
  int dtype;
  size_t esize;
};

ea_status check_params(const ea_params* p) {
  if (!std::isfinite(p->alpha) || !(p->alpha > 1.0f)) return EA_ERR_INVALID_ARG;
  if (!std::isfinite(p->scale) || !(p->scale > 0.0f)) return EA_ERR_INVALID_ARG;
  if (p->causal != 0 && p->causal != 1) return EA_ERR_INVALID_ARG;
  if (p->need_bwd != 0 && p->need_bwd != 1) return EA_ERR_INVALID_ARG;
  if (p->max_iter < 0 || p->max_iter > MAX_ITER_CAP) return EA_ERR_INVALID_ARG;
  if (!std::isfinite(p->tol) || p->tol < 0.0f) return EA_ERR_INVALID_ARG;
  return EA_OK;
}

ea_status check_shape(const ea_shape* s, const ea_params* p, Dims* out) {
  if (!s || !p) return EA_ERR_INVALID_ARG;
  if (s->batch < 1 || s->heads < 1 || s->seqlen < 1 || s->head_dim < 1) return EA_ERR_INVALID_ARG;
  if (s->dtype != EA_BF16 && s->dtype != EA_F32) return EA_ERR_UNSUPPORTED;
  if (s->head_dim != 64 && s->head_dim != 128) return EA_ERR_UNSUPPORTED;
  if (s->seqlen > MAX_SEQLEN) return EA_ERR_UNSUPPORTED;
  const ea_status st = check_params(p);
  if (st != EA_OK) return st;
  const int64_t BH = (int64_t)s->batch * s->heads;
  const int64_t n = s->seqlen;
  const int64_t T = (n + 63) / 64;
  // grid sizes and in-kernel offsets use 32-bit block counts
  if (BH * ((n + 63) / 64) > (int64_t)INT32_MAX / 2) return EA_ERR_UNSUPPORTED;
  out->BH = BH;
  out->n = n;
  out->d = s->head_dim;
  out->T = T;
  out->elems = BH * n * s->head_dim;
  out->dtype = s->dtype;
  out->esize = s->dtype == EA_BF16 ? 2 : 4;
  return EA_OK;
}

// delta, one fp32 per row
size_t bwd_ws_bytes(const Dims& d) { return (size_t)(d.BH * d.n) * 4; }

// One cache slot per solver tile (256 rows on the masked path, 128 rows in
// the no-mask fused forward), at most MAX_SOLVE_SLOTS of the masked path's
// size: two co-resident workgroups per CU of a 256-CU MI355X.  With fewer
// slots than tiles the solvers run one workgroup per slot, each solving
// tiles in turn, so the workspace does not grow with B * H * n.  The masked
// path's sizing covers both.
constexpr int64_t MAX_SOLVE_SLOTS = 512;
int64_t solve_tiles(const Dims& d) { return d.BH * ((d.n + SOLVE_ROWS - 1) / SOLVE_ROWS); }
int64_t cache_tiles(const Dims& d) { return d.BH * ((d.n + TAU_ROWS - 1) / TAU_ROWS); }
int64_t solve_slots(const Dims& d) {
  return solve_tiles(d) < MAX_SOLVE_SLOTS ? solve_tiles(d) : MAX_SOLVE_SLOTS;
}
static_assert(SOLVE_ROWS == 2 * TAU_ROWS && SOLVE_SLOT_BYTES >= 2 * TAU_SLOT_BYTES,
              "a masked-path slot covers two fused-forward slots");

void fill_sizes(const Dims& d, ea_sizes* z) {
  z->tau = (size_t)(d.BH * d.n) * 4;
  z->o2 = (size_t)d.elems * 4;
  z->block_mask = (size_t)(d.BH * d.T * d.T);
  z->q_count = (size_t)(d.BH * d.T) * 4;
  z->q_index = (size_t)(d.BH * d.T * d.T) * 4;
  z->k_count = z->q_count;
  z->k_index = z->q_index;
  z->stats = (size_t)(2 * d.BH * d.T) * 4;
  z->ws_fwd = (size_t)solve_slots(d) * SOLVE_SLOT_BYTES;
  z->ws_bwd = bwd_ws_bytes(d);
  z->tau_lo = d.dtype == EA_F32 ? (size_t)(d.BH * d.n) * 4 : 0;
}

bool tensor_ok(const void* p) { return p && aligned(p, 16); }
bool small_ok(const void* p) { return p && aligned(p, 4); }

ea_status check_tables(const ea_residuals* r, const Dims& d) {
  if (!r) return EA_ERR_INVALID_ARG;
  if (!small_ok(r->tau) || !r->block_mask || !small_ok(r->q_count) || !small_ok(r->q_index) ||
      !small_ok(r->k_count) || !small_ok(r->k_index))
    return EA_ERR_INVALID_ARG;
  if (r->stats && !aligned(r->stats, 4)) return EA_ERR_INVALID_ARG;
  if (d.dtype == EA_F32 && !small_ok(r->tau_lo)) return EA_ERR_INVALID_ARG;
  return EA_OK;
}

// fp64 parameters of the fp32 inputs' refinement, from the fp32 values given
double c64_of(const ea_params* p) { return ((double)p->alpha - 1.0) * (double)p->scale; }
double g64_of(const ea_params* p) { return 1.0 / ((double)p->alpha - 1.0); }
const float* tau_lo_of(const ea_residuals* r, const Dims& d) {
  return d.dtype == EA_F32 ? r->tau_lo : nullptr;
}

// HIP error behind the calling thread's most recent EA_ERR_HIP.
thread_local hipError_t last_hip_error = hipSuccess;

// Checks shared by the row-wise entry points; fills the kernel arguments.
ea_status prep_rows(int64_t rows, int32_t n, ea_dtype dtype, const ea_params* params,
                    const void* s, RowsArgs* ra) {
  if (!params) return EA_ERR_INVALID_ARG;
  ea_status st = check_params(params);
  if (st != EA_OK) return st;
  if (rows < 1 || n < 1) return EA_ERR_INVALID_ARG;
  if (dtype != EA_BF16 && dtype != EA_F32) return EA_ERR_UNSUPPORTED;
  if (n > MAX_ROW_LEN || rows > (int64_t)INT32_MAX) return EA_ERR_UNSUPPORTED;
  if (!tensor_ok(s)) return EA_ERR_INVALID_ARG;
  *ra = RowsArgs{};
  ra->s = s;
  ra->rows = rows;
  ra->n = n;
  ra->alpha = params->alpha;
  ra->gamma = 1.0f / (params->alpha - 1.0f);
  ra->scale = params->scale;
  ra->c = (params->alpha - 1.0f) * params->scale;
  ra->tol = params->tol;
  ra->max_iter = params->max_iter;
  ra->gk = gamma_kind(params->alpha);
  return EA_OK;
}

ea_status from_hip(hipError_t e) {
  if (e == hipSuccess) return EA_OK;
  last_hip_error = e;
  return EA_ERR_HIP;
}

constexpr int MAX_DEVICES = 64;
std::mutex scratch_mutex;
float* scratch_ptr[MAX_DEVICES] = {};

// Device address of `scratch` on the device that `stream` belongs to (the
// current device for the null stream); null on failure with *err set.
float* scratch_for(hipStream_t stream, hipError_t* err) {
  int dev = 0;
  *err = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (*err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= MAX_DEVICES) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (scratch_ptr[dev]) return scratch_ptr[dev];
  int cur = 0;
  if ((*err = hipGetDevice(&cur)) != hipSuccess) return nullptr;
  if (cur != dev && (*err = hipSetDevice(dev)) != hipSuccess) return nullptr;
  void* p = nullptr;
  *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (cur != dev) {
    const hipError_t e2 = hipSetDevice(cur);
    if (*err == hipSuccess) *err = e2;
  }
  if (*err != hipSuccess) return nullptr;
  scratch_ptr[dev] = static_cast<float*>(p);
  return scratch_ptr[dev];
}

}  // namespace
}  // namespace ea

using namespace ea;

extern "C" {

void entmax_attn_default_params(ea_params* p) {
  if (!p) return;
  p->alpha = 1.5f;
  p->scale = 0.125f;
  p->causal = 0;
  p->max_iter = DEFAULT_MAX_ITER;
  p->tol = DEFAULT_TOL;
  p->need_bwd = 1;
}

ea_status entmax_attn_sizes(const ea_shape* shape, const ea_params* params, ea_sizes* out) {
  Dims d;
  ea_status st = check_shape(shape, params, &d);
  if (st != EA_OK) return st;
  if (!out) return EA_ERR_INVALID_ARG;
  fill_sizes(d, out);
  return EA_OK;
}

namespace {

// Checks shared by the forward entry points; fills the kernel arguments.
ea_status prep_fwd(const ea_shape* shape, const ea_params* params, const void* q, const void* k,
                   const void* v, void* o, const ea_residuals* res, const void* workspace,
                   Dims* d) {
  ea_status st = check_shape(shape, params, d);
  if (st != EA_OK) return st;
  if (workspace && !aligned(workspace, 16)) return EA_ERR_INVALID_ARG;
  if (!tensor_ok(q) || !tensor_ok(k) || !tensor_ok(v) || !tensor_ok(o)) return EA_ERR_INVALID_ARG;
  if ((st = check_tables(res, *d)) != EA_OK) return st;
  if (params->need_bwd && !tensor_ok(res->o2)) return EA_ERR_INVALID_ARG;
  return EA_OK;
}

ea_status run_fwd_stage(int stage, const Dims& d, const ea_params* params, const void* q,
                        const void* k, const void* v, void* o, const ea_residuals* res,
                        void* workspace, size_t ws_bytes, hipStream_t s) {
  const float c = (params->alpha - 1.0f) * params->scale;
  const float gamma = 1.0f / (params->alpha - 1.0f);
  const int gk = gamma_kind(params->alpha);
  if (stage == 0) {
    // The cache is optional: tiles without a slot (all of them when there is
    // no workspace) stream K on every solver pass.
    int64_t slots = workspace ? (int64_t)(ws_bytes / SOLVE_SLOT_BYTES) : 0;
    const int64_t most = solve_tiles(d);
    if (slots > most) slots = most;
    void* cand = slots > 0 ? workspace : nullptr;
    TauArgs ta{q, k, res->tau, res->block_mask, res->stats, nullptr, nullptr, nullptr, cand,
               SOLVE_QUAD_CAP, (int)slots, /*tile0=*/0,
               (int)d.BH, (int)d.n, (int)d.T, c, params->alpha, gamma, params->causal,
               params->max_iter, params->tol, gk,
               const_cast<float*>(tau_lo_of(res, d)), c64_of(params), g64_of(params),
               res->q_count, res->q_index};
    return from_hip(launch_tau(ta, d.dtype, (int)d.d, s));
  }
  FwdArgs fa{q, k, v, o, params->need_bwd ? res->o2 : nullptr, res->tau, res->q_count,
             res->q_index, (int)d.BH, (int)d.n, (int)d.T, c, gamma, params->causal, gk,
             tau_lo_of(res, d), c64_of(params), g64_of(params),
             res->block_mask, res->k_count, res->k_index};
  return from_hip(launch_fwd(fa, d.dtype, (int)d.d, params->need_bwd != 0, s));
}

// Checks of the backward's tensors and residuals (not its workspace).
ea_status prep_bwd_args(const ea_shape* shape, const ea_params* params, const void* q,
                        const void* k, const void* v, const void* dout, const ea_residuals* res,
                        const float* dq, const float* dk, const float* dv, Dims* d) {
  ea_status st = check_shape(shape, params, d);
  if (st != EA_OK) return st;
  if (!tensor_ok(q) || !tensor_ok(k) || !tensor_ok(v) || !tensor_ok(dout)) return EA_ERR_INVALID_ARG;
  if (!tensor_ok(dq) || !tensor_ok(dk) || !tensor_ok(dv)) return EA_ERR_INVALID_ARG;
  if ((st = check_tables(res, *d)) != EA_OK) return st;
  if (!tensor_ok(res->o2)) return EA_ERR_INVALID_ARG;
  return EA_OK;
}

ea_status prep_bwd(const ea_shape* shape, const ea_params* params, const void* q, const void* k,
                   const void* v, const void* dout, const ea_residuals* res, const float* dq,
                   const float* dk, const float* dv, const void* workspace, size_t ws_bytes,
                   Dims* d) {
  ea_status st = prep_bwd_args(shape, params, q, k, v, dout, res, dq, dk, dv, d);
  if (st != EA_OK) return st;
  if (!workspace || !aligned(workspace, 16)) return EA_ERR_INVALID_ARG;
  if (ws_bytes < bwd_ws_bytes(*d)) return EA_ERR_WORKSPACE;
  return EA_OK;
}

ea_status run_bwd_stage(int stage, const Dims& d, const ea_params* params, const void* q,
                        const void* k, const void* v, const void* dout, const ea_residuals* res,
                        float* dq, float* dk, float* dv, void* workspace, hipStream_t s) {
  float* delta = static_cast<float*>(workspace);
  if (stage == 0) {
    DeltaArgs da{dout, res->o2, delta, d.BH * d.n};
    return from_hip(launch_delta(da, d.dtype, (int)d.d, s));
  }
  const float c = (params->alpha - 1.0f) * params->scale;
  const float gamma = 1.0f / (params->alpha - 1.0f);
  BwdArgs ba{q, k, v, dout, res->tau, delta, res->q_count, res->q_index, res->k_count,
             res->k_index, dq, dk, dv, (int)d.BH, (int)d.n, (int)d.T, c, gamma,
             params->scale, params->causal, gamma_kind(params->alpha), tau_lo_of(res, d),
             c64_of(params), g64_of(params)};
  if (stage == 1) return from_hip(launch_bwd_dkdv(ba, d.dtype, (int)d.d, s));
  return from_hip(launch_bwd_dq(ba, d.dtype, (int)d.d, s));
}

}  // namespace

ea_status entmax_attn_fwd(const ea_shape* shape, const ea_params* params, const void* q,
                          const void* k, const void* v, void* o, const ea_residuals* res,
                          void* workspace, size_t ws_bytes, void* stream) {
  Dims d;
  ea_status st = prep_fwd(shape, params, q, k, v, o, res, workspace, &d);
  if (st != EA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int stage = 0; stage < 2; ++stage)
    if ((st = run_fwd_stage(stage, d, params, q, k, v, o, res, workspace, ws_bytes, s)) != EA_OK)
      return st;
  return EA_OK;
}

ea_status entmax_attn_fwd_stage(int stage, const ea_shape* shape, const ea_params* params,
                                const void* q, const void* k, const void* v, void* o,
                                const ea_residuals* res, void* workspace, size_t ws_bytes,
                                void* stream) {
  if (stage < 0 || stage > 1) return EA_ERR_INVALID_ARG;
  Dims d;
  ea_status st = prep_fwd(shape, params, q, k, v, o, res, workspace, &d);
  if (st != EA_OK) return st;
  return run_fwd_stage(stage, d, params, q, k, v, o, res, workspace, ws_bytes,
                       static_cast<hipStream_t>(stream));
}

ea_status entmax_attn_bwd(const ea_shape* shape, const ea_params* params, const void* q,
                          const void* k, const void* v, const void* dout,
                          const ea_residuals* res, float* dq, float* dk, float* dv,
                          void* workspace, size_t ws_bytes, void* stream) {
  Dims d;
  ea_status st = prep_bwd(shape, params, q, k, v, dout, res, dq, dk, dv, workspace, ws_bytes, &d);
  if (st != EA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int stage = 0; stage < 3; ++stage)
    if ((st = run_bwd_stage(stage, d, params, q, k, v, dout, res, dq, dk, dv, workspace, s)) != EA_OK)
      return st;
  return EA_OK;
}

ea_status entmax_attn_bwd_stage(int stage, const ea_shape* shape, const ea_params* params,
                                const void* q, const void* k, const void* v, const void* dout,
                                const ea_residuals* res, float* dq, float* dk, float* dv,
                                void* workspace, size_t ws_bytes, void* stream) {
  if (stage < 0 || stage > 2) return EA_ERR_INVALID_ARG;
  Dims d;
  ea_status st = prep_bwd(shape, params, q, k, v, dout, res, dq, dk, dv, workspace, ws_bytes, &d);
  if (st != EA_OK) return st;
  return run_bwd_stage(stage, d, params, q, k, v, dout, res, dq, dk, dv, workspace,
                       static_cast<hipStream_t>(stream));
}

ea_status entmax_attn_bwd_noalloc(const ea_shape* shape, const ea_params* params, const void* q,
                                  const void* k, const void* v, const void* dout,
                                  const ea_residuals* res, float* dq, float* dk, float* dv,
                                  void* stream) {
  Dims d;
  ea_status st = check_shape(shape, params, &d);
  if (st != EA_OK) return st;
  if (d.BH * d.n > (int64_t)EA_NOALLOC_MAX_ROWS) return EA_ERR_UNSUPPORTED;
  if ((st = prep_bwd_args(shape, params, q, k, v, dout, res, dq, dk, dv, &d)) != EA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  float* delta = scratch_for(s, &e);
  if (!delta) return from_hip(e);
  for (int stage = 0; stage < 3; ++stage)
    if ((st = run_bwd_stage(stage, d, params, q, k, v, dout, res, dq, dk, dv, delta, s)) != EA_OK)
      return st;
  return EA_OK;
}

ea_status entmax_rows_fwd(int64_t rows, int32_t n, ea_dtype dtype, const ea_params* params,
                          const void* s, float* p, float* tau, void* stream) {
  RowsArgs ra;
  ea_status st = prep_rows(rows, n, dtype, params, s, &ra);
  if (st != EA_OK) return st;
  if (!tensor_ok(p) || !tensor_ok(tau)) return EA_ERR_INVALID_ARG;
  ra.p = p;
  ra.tau = tau;
  return from_hip(launch_rows_fwd(ra, dtype, static_cast<hipStream_t>(stream)));
}

ea_status entmax_rows_bwd(int64_t rows, int32_t n, ea_dtype dtype, const ea_params* params,
                          const void* s, const float* tau, const float* dp, float* ds,
                          void* stream) {
  RowsArgs ra;
  ea_status st = prep_rows(rows, n, dtype, params, s, &ra);
  if (st != EA_OK) return st;
  if (!tensor_ok(tau) || !tensor_ok(dp) || !tensor_ok(ds)) return EA_ERR_INVALID_ARG;
  ra.tau = const_cast<float*>(tau);  // read only by the backward kernel
  ra.dp = dp;
  ra.ds = ds;
  return from_hip(launch_rows_bwd(ra, dtype, static_cast<hipStream_t>(stream)));
}

ea_status entmax_attn_fwd_dense(const ea_shape* shape, const ea_params* params, const void* q,
                                const void* k, const void* v, void* o, float* tau, float* tau_lo,
                                float* o2, void* workspace, size_t ws_bytes, void* stream) {
  Dims d;
  ea_status st = check_shape(shape, params, &d);
  if (st != EA_OK) return st;
  if (!tensor_ok(q) || !tensor_ok(k) || !tensor_ok(v) || !tensor_ok(o)) return EA_ERR_INVALID_ARG;
  if (!small_ok(tau)) return EA_ERR_INVALID_ARG;
  if (d.dtype == EA_F32 && !small_ok(tau_lo)) return EA_ERR_INVALID_ARG;
  if (params->need_bwd && !tensor_ok(o2)) return EA_ERR_INVALID_ARG;
  if (workspace && !aligned(workspace, 16)) return EA_ERR_INVALID_ARG;
  int64_t slots = workspace ? (int64_t)(ws_bytes / TAU_SLOT_BYTES) : 0;
  if (slots > cache_tiles(d)) slots = cache_tiles(d);
  void* cand = slots > 0 ? workspace : nullptr;
  const float c = (params->alpha - 1.0f) * params->scale;
  const float gamma = 1.0f / (params->alpha - 1.0f);
  TauArgs ta{q, k, tau, nullptr, nullptr, v, o, params->need_bwd ? o2 : nullptr, cand,
             TAU_CACHE_CAP, (int)slots, /*tile0=*/0, (int)d.BH, (int)d.n, (int)d.T, c,
             params->alpha, gamma,
             params->causal, params->max_iter, params->tol, gamma_kind(params->alpha),
             d.dtype == EA_F32 ? tau_lo : nullptr, c64_of(params), g64_of(params)};
  return from_hip(launch_tau_fused(ta, d.dtype, (int)d.d, static_cast<hipStream_t>(stream)));
}

ea_status entmax_attn_bwd_dense(const ea_shape* shape, const ea_params* params, const void* q,
                                const void* k, const void* v, const void* dout, const float* tau,
                                const float* tau_lo, const float* o2, float* dq, float* dk,
                                float* dv, void* workspace, size_t ws_bytes, void* stream) {
  Dims d;
  ea_status st = check_shape(shape, params, &d);
  if (st != EA_OK) return st;
  if (!tensor_ok(q) || !tensor_ok(k) || !tensor_ok(v) || !tensor_ok(dout)) return EA_ERR_INVALID_ARG;
  if (!tensor_ok(dq) || !tensor_ok(dk) || !tensor_ok(dv)) return EA_ERR_INVALID_ARG;
  if (!small_ok(tau) || !tensor_ok(o2)) return EA_ERR_INVALID_ARG;
  if (d.dtype == EA_F32 && !small_ok(tau_lo)) return EA_ERR_INVALID_ARG;
  if (!workspace || !aligned(workspace, 16)) return EA_ERR_INVALID_ARG;
  if (ws_bytes < bwd_ws_bytes(d)) return EA_ERR_WORKSPACE;
  // no tables: the kernels visit every valid block
  ea_residuals res{};
  res.tau = const_cast<float*>(tau);
  res.tau_lo = const_cast<float*>(tau_lo);
  res.o2 = const_cast<float*>(o2);
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int stage = 0; stage < 3; ++stage)
    if ((st = run_bwd_stage(stage, d, params, q, k, v, dout, &res, dq, dk, dv, workspace, s)) != EA_OK)
      return st;
  return EA_OK;
}

const char* entmax_attn_status_string(ea_status s) {
  switch (s) {
    case EA_OK: return "ok";
    case EA_ERR_INVALID_ARG: return "invalid argument";
    case EA_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case EA_ERR_WORKSPACE: return "workspace too small";
    case EA_ERR_HIP: return "HIP launch failure";
  }
  return "unknown status";
}

const char* entmax_attn_last_hip_error(void) {
  return last_hip_error == hipSuccess ? "" : hipGetErrorName(last_hip_error);
}

}  // extern "C"
