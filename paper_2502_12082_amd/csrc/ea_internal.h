// ea_internal.h -- launch interface between the C ABI (ea_api.hip) and the
// kernel translation units.  Host-side only; no torch, no exceptions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ea {

// Largest sequence length the kernels accept (the solver keeps one byte per
// (wave, key block) of mask state in LDS).
constexpr int MAX_SEQLEN = 131072;
constexpr int MAX_KEY_BLOCKS = MAX_SEQLEN / 64;

// Which specialisation of the per-element map: gamma = 1/(alpha-1) in
// {1, 2, 4} run without transcendentals; 0 means general alpha.
int gamma_kind(float alpha);

// One cached score of the no-mask forward's solver: the raw score
// s = <q_i, k_j> (the solver forms x - tau from it exactly as in a streamed
// evaluation) and the key j.
struct alignas(8) CandEntry {
  float s;
  int32_t j;  // key index; its key block is j / 64
};

// Workgroup geometry (rows and threads per workgroup) of the masked path's
// solver and of the no-mask fused forward.  Each row has two candidate
// lists (one per half of every key block), of `cap` entries each.
constexpr int SOLVE_ROWS = 256;
constexpr int SOLVE_THREADS = 256;
constexpr int TAU_ROWS = 128;
constexpr int TAU_THREADS = 256;

// The masked path's solver caches quads: the four raw scores of four
// consecutive keys 4 m .. 4 m + 3 that one lane holds for one row (16 bytes),
// with m as a 16-bit key (2 bytes, in an array of their own).  Its first
// evaluation copies the scores above the bracket's lower end into lists of
// single scores (4 bytes, and their key blocks, 2 bytes).  A slot holds
// `cap` quads and `cap` singles in each of the 2 * SOLVE_THREADS lists of a
// workgroup.
constexpr size_t SOLVE_QUAD_BYTES = 16 + 2;
constexpr size_t SOLVE_SINGLE_BYTES = 4 + 2;
constexpr size_t solve_slot_bytes(int cap) {
  return (size_t)cap * 2 * SOLVE_THREADS * (SOLVE_QUAD_BYTES + SOLVE_SINGLE_BYTES);
}
static_assert(MAX_SEQLEN / 4 <= 65536, "a quad's key fits 16 bits");

struct TauArgs {
  const void* q;
  const void* k;
  float* tau;         // [BH, n]
  uint8_t* mask;      // [BH, T, T]
  int32_t* stats;     // [2, BH, T] K passes and evaluations for each 64-row query block, or null
  // no-mask mode only (mask, stats null): O and, when training, O2 are
  // accumulated by the solver kernel itself once tau is known
  const void* v;
  void* o;            // [BH, n, D] input dtype
  float* o2;          // [BH, n, D] fp32, or null (inference)
  void* cand;         // candidate cache: one slot per workgroup (quads or CandEntry lists), or null
  int cap;            // entries (quads for the masked path) per list
  int slots;          // cache slots (workgroup b of a launch uses slot b)
  int tile0;          // first tile of this launch (workgroup b solves tile tile0 + b)
  int BH, n, T;
  float c;            // (alpha - 1) * scale
  float alpha, gamma;
  int causal, max_iter;
  float tol;
  int gk;             // gamma_kind(alpha)
  // fp32 inputs, general alpha: tau is refined in fp64 and written as
  // tau + tau_lo ([BH, n]); c64, g64 are (alpha - 1) * scale and 1/(alpha - 1)
  // in fp64 from the same fp32 parameters
  float* tau_lo;
  double c64, g64;
  // masked path: the row tables of the mask (Q_i of every query block),
  // written with it
  int32_t* q_count;   // [BH, T]
  int32_t* q_index;   // [BH, T, T]
};

struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;                // [BH, n, D] input dtype
  float* o2;              // [BH, n, D] fp32, train only
  const float* tau;
  const int32_t* q_count;
  const int32_t* q_index;
  int BH, n, T;
  float c, gamma;
  int causal;
  int gk;
  const float* tau_lo;  // fp32 inputs, general alpha: low part of tau (or null: 0)
  double c64, g64;
  // the column tables (K_j of every key block), built by extra workgroups of
  // the same launch from the mask
  const uint8_t* mask;  // [BH, T, T]
  int32_t* k_count;     // [BH, T]
  int32_t* k_index;     // [BH, T, T]
};

struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* dout;
  const float* tau;
  const float* delta;     // [BH, n]
  const int32_t* q_count;
  const int32_t* q_index;
  const int32_t* k_count;
  const int32_t* k_index;
  float *dq, *dk, *dv;
  int BH, n, T;
  float c, gamma, scale;
  int causal;
  int gk;
  const float* tau_lo;  // fp32 inputs, general alpha: low part of tau (or null: 0)
  double c64, g64;
};

struct DeltaArgs {
  const void* dout;
  const float* o2;
  float* delta;
  int64_t rows;
};

// Row-wise alpha-entmax of a materialized [rows, n] score matrix.
struct RowsArgs {
  const void* s;      // [rows, n] scores, input dtype
  float* p;           // [rows, n] probabilities (forward output)
  float* tau;         // [rows] thresholds (forward output, backward input)
  const float* dp;    // [rows, n] gradient of p (backward input)
  float* ds;          // [rows, n] gradient of s (backward output)
  int64_t rows;
  int n;
  float c;            // (alpha - 1) * scale
  float alpha, gamma, scale, tol;
  int max_iter, gk;
};

// Largest row the row-wise kernels hold in registers.
constexpr int MAX_ROW_LEN = 32768;

// Each launcher picks the instantiation for (dtype: 0 bf16 / 1 fp32, head_dim,
// gamma kind) and returns the launch status.
// Launches `kernel` with its one argument struct and returns the launch's own
// status (not an error left behind by earlier HIP calls on this thread).
template <typename A>
inline hipError_t launch_kernel(void (*kernel)(A), dim3 grid, dim3 block, hipStream_t s, A a) {
  void* args[] = {&a};
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, args, 0, s);
}

hipError_t launch_tau(const TauArgs& a, int dtype, int head_dim, hipStream_t s);
// The no-mask forward: tau, then O (and O2 if a.o2) in the same kernel.
hipError_t launch_tau_fused(const TauArgs& a, int dtype, int head_dim, hipStream_t s);
hipError_t launch_fwd(const FwdArgs& a, int dtype, int head_dim, bool train, hipStream_t s);
hipError_t launch_delta(const DeltaArgs& a, int dtype, int head_dim, hipStream_t s);
hipError_t launch_bwd_dkdv(const BwdArgs& a, int dtype, int head_dim, hipStream_t s);
hipError_t launch_bwd_dq(const BwdArgs& a, int dtype, int head_dim, hipStream_t s);
hipError_t launch_rows_fwd(const RowsArgs& a, int dtype, hipStream_t s);
hipError_t launch_rows_bwd(const RowsArgs& a, int dtype, hipStream_t s);

}  // namespace ea
