// ea_rows.hip -- row-wise alpha-entmax of a materialized score matrix.
//
// Forward (Sec. 3.1, Algorithm 1): for each row s of length n,
// x = (alpha-1) * scale * s, tau is the root of f(tau) = sum_j [x_j -
// tau]_+^gamma - 1 (Eq. 3) found by the hybrid Halley-bisection iteration
// (Eq. 4, 5, with f', f'' of Eq. 6, 7), and p_j = [x_j - tau]_+^gamma (Eq. 2).
// Backward: with u_j = [x_j - tau]_+^(gamma-1) on the support, the Jacobian
// of p with respect to s is scale * (Diag(u) - u u^T / sum u) (Sec. 3.2.2;
// (alpha-1) gamma = 1), so ds = scale * u (dp - <u, dp> / sum u).
//
// Layout: NT threads per row (a workgroup of 256, or in the forward one
// wave of 64 for rows of up to 2048 elements); thread t keeps elements
// 4 (t + NT w) + e, w < VPT / 4, e < 4, in registers (16-byte accesses when
// n is a multiple of 8), so the row is read once and every evaluation of
// the iteration runs from registers, with one reduction over the row's
// threads per evaluation.  The forward runs rows of more than 4096 elements
// in persistent workgroups that load their next row while iterating on the
// current one.  The update rules are
// those of the attention solver: the bracket test with its rounding slack,
// the Newton lower bound for gamma >= 1 and the midpoint safeguard for
// gamma < 1.
#include <type_traits>

#include "ea_common.h"
#include "ea_internal.h"

namespace ea {

namespace {

constexpr int ROW_NT = 256;

// Workgroup barrier for LDS traffic only: unlike __syncthreads it does not
// wait for this wave's global loads, so a row prefetched into registers
// stays in flight across the reductions of the current row.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <bool LDS_ONLY>
__device__ __forceinline__ void row_barrier() {
  if constexpr (LDS_ONLY)
    lds_barrier();
  else
    __syncthreads();
}

struct Sums {
  float a, b, c;
  int k;
};

// Workgroup totals of (a, b, c, k); every thread receives them.  The order
// of the additions is fixed, so results are deterministic.
template <bool LDS_ONLY = false, int NT = ROW_NT>
__device__ __forceinline__ Sums wg_sum(Sums v, float* sh) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    v.a += __shfl_xor(v.a, o);
    v.b += __shfl_xor(v.b, o);
    v.c += __shfl_xor(v.c, o);
    v.k += __shfl_xor(v.k, o);
  }
  const int w = wave_id();
  if (lane_id() == 0) {
    sh[4 * w + 0] = v.a;
    sh[4 * w + 1] = v.b;
    sh[4 * w + 2] = v.c;
    sh[4 * w + 3] = __int_as_float(v.k);
  }
  row_barrier<LDS_ONLY>();
  Sums t{0.f, 0.f, 0.f, 0};
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    t.a += sh[4 * i + 0];
    t.b += sh[4 * i + 1];
    t.c += sh[4 * i + 2];
    t.k += __float_as_int(sh[4 * i + 3]);
  }
  row_barrier<LDS_ONLY>();  // sh is reused by the next reduction
  return t;
}

template <bool LDS_ONLY = false>
__device__ __forceinline__ float wg_max(float v, float* sh) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  if (lane_id() == 0) sh[wave_id()] = v;
  row_barrier<LDS_ONLY>();
  float t = sh[0];
#pragma unroll
  for (int i = 1; i < ROW_NT / 64; ++i) t = fmaxf(t, sh[i]);
  row_barrier<LDS_ONLY>();
  return t;
}

// Element held in slot v of the calling thread: groups of 4 consecutive
// elements, so that rows whose length is a multiple of 8 move in 16-byte
// (fp32) or 8-byte (bf16) accesses.
template <int VPT, int NT = ROW_NT>
__device__ __forceinline__ int row_elem(int v, int t = (int)threadIdx.x) {
  return 4 * (t + NT * (v / 4)) + (v % 4);
}

// The raw values of a row held for the prefetch: one 16-byte (fp32) or
// 8-byte (bf16) group of four elements per four slots, loaded through a
// buffer resource over the row, so that groups past its end read 0 and the
// loads need no branches (rows of a multiple of 8 elements; a branch would
// make the compiler wait for each load to unpack it).
template <typename E, int VPT>
struct RawRow {
  using V = typename std::conditional<sizeof(E) == 4, f32x4, bf16x4>::type;
  V g[VPT / 4];

  __device__ __forceinline__ void load(const E* row, int n) {
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(const_cast<E*>(row), (uint32_t)n * (uint32_t)sizeof(E));
#pragma unroll
    for (int g4 = 0; g4 < VPT / 4; ++g4) {
      const uint32_t off = (uint32_t)row_elem<VPT>(4 * g4) * (uint32_t)sizeof(E);
      if constexpr (sizeof(E) == 4)
        g[g4] = __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
      else
        g[g4] = __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
    }
  }

  // x = c * value, -inf past the end of the row
  __device__ __forceinline__ void scale(int n, float c, float (&x)[VPT]) const {
#pragma unroll
    for (int g4 = 0; g4 < VPT / 4; ++g4)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        x[4 * g4 + e] = row_elem<VPT>(4 * g4 + e) < n ? c * (float)g[g4][e] : -INFINITY;
  }
};

template <typename E, int VPT, int NT = ROW_NT>
__device__ __forceinline__ void load_row(const E* s, int n, float c, float (&x)[VPT], int t = (int)threadIdx.x) {
  static_assert(VPT % 4 == 0, "slots come in groups of 4");
  const bool vec = (n % 8) == 0;
#pragma unroll
  for (int g4 = 0; g4 < VPT / 4; ++g4) {
    const int j0 = row_elem<VPT, NT>(4 * g4, t);
    if (vec && j0 < n) {
      if constexpr (sizeof(E) == 4) {
        const f32x4 v4 = *reinterpret_cast<const f32x4*>(s + j0);
#pragma unroll
        for (int e = 0; e < 4; ++e) x[4 * g4 + e] = c * v4[e];
      } else {
        const bf16x4 v4 = *reinterpret_cast<const bf16x4*>(s + j0);
#pragma unroll
        for (int e = 0; e < 4; ++e) x[4 * g4 + e] = c * (float)v4[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        x[4 * g4 + e] = j0 + e < n ? c * (float)s[j0 + e] : -INFINITY;  // padding: [x - tau]_+ = 0
    }
  }
}

// Stores slot values y to row r (length n) in the same element order.
template <int VPT, int NT = ROW_NT>
__device__ __forceinline__ void store_row(float* r, int n, const float (&y)[VPT], int t = (int)threadIdx.x) {
  const bool vec = (n % 8) == 0;
#pragma unroll
  for (int g4 = 0; g4 < VPT / 4; ++g4) {
    const int j0 = row_elem<VPT, NT>(4 * g4, t);
    if (vec && j0 < n) {
      *reinterpret_cast<f32x4*>(r + j0) = f32x4{y[4 * g4], y[4 * g4 + 1], y[4 * g4 + 2], y[4 * g4 + 3]};
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j0 + e < n) r[j0 + e] = y[4 * g4 + e];
    }
  }
}

// Reductions over the threads that hold one row: a workgroup through LDS
// (LDS_ONLY: with a barrier that leaves global loads in flight), or a single
// wave through lane exchanges alone.  Every thread receives the totals; the
// exchanges add commutative pairs, so all lanes hold the same bits.
template <bool LDS_ONLY>
struct WgRed {
  float* sh;
  __device__ __forceinline__ float max(float v) const { return wg_max<LDS_ONLY>(v, sh); }
  __device__ __forceinline__ Sums sum(Sums v) const { return wg_sum<LDS_ONLY>(v, sh); }
};

struct WaveRed {
  __device__ __forceinline__ float max(float v) const {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
  }
  __device__ __forceinline__ Sums sum(Sums v) const {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      v.a += __shfl_xor(v.a, o);
      v.b += __shfl_xor(v.b, o);
      v.c += __shfl_xor(v.c, o);
      v.k += __shfl_xor(v.k, o);
    }
    return v;
  }
};

// Algorithm 1 on one row: tau for the scaled scores x this thread holds
// (-inf past the end of the row), the row's other values held by the
// threads that `red` reduces over.
template <int VPT, int GK, typename Red>
__device__ __forceinline__ float row_tau(const float (&x)[VPT], int n, const RowsArgs& a, const Red& red) {
  const float g = a.gamma;
  float mx = -INFINITY;
#pragma unroll
  for (int v = 0; v < VPT; ++v) mx = fmaxf(mx, x[v]);
  const float m = red.max(mx);

  // Algorithm 1: bracket [m - 1, m - n^(1-alpha)], first tau at its midpoint
  float lo = m - 1.f, hi = m - powf((float)n, 1.f - a.alpha);
  float tau = 0.5f * (lo + hi);
  const bool newton_bound = g >= 1.f;
  float f_prev = INFINITY;
  for (int it = 0;; ++it) {
    Sums t{0.f, 0.f, 0.f, 0};
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const float zp = __builtin_amdgcn_fmed3f(x[v] - tau, 0.f, 1.f);
      if constexpr (GK == 1) {
        t.a += zp;
        t.k += in_support(zp);
      } else if constexpr (GK == 2) {
        t.a = fmaf(zp, zp, t.a);
        t.b += zp;
        t.k += in_support(zp);
      } else if constexpr (GK == 4) {
        const float z2 = zp * zp;
        t.a = fmaf(z2, z2, t.a);
        t.b = fmaf(z2, zp, t.b);
        t.c += z2;
      } else {
        if (zp > 0.f) {
          const float l = __log2f(zp);
          t.a += exp2f(g * l);
          t.b += exp2f((g - 1.f) * l);
          t.c += exp2f((g - 2.f) * l);
        }
      }
    }
    const Sums tot = red.sum(t);
    const float f = tot.a - 1.f;  // Eq. 3
    float f1, f2;                 // Eq. 6, 7
    if constexpr (GK == 1) {
      f1 = -(float)tot.k;
      f2 = 0.f;
    } else if constexpr (GK == 2) {
      f1 = -2.f * tot.b;
      f2 = 2.f * (float)tot.k;
    } else if constexpr (GK == 4) {
      f1 = -4.f * tot.b;
      f2 = 12.f * tot.c;
    } else {
      f1 = -g * tot.b;
      f2 = g * (g - 1.f) * tot.c;
    }
    if (fabsf(f) <= a.tol || it >= a.max_iter) break;
    if (f < 0.f)  // B_f, Eq. 4
      hi = tau;
    else
      lo = tau;
    const float slack = 1e-6f * fmaxf(1.f, fmaxf(fabsf(lo), fabsf(hi)));
    if (newton_bound && f1 < 0.f) lo = fminf(fmaxf(lo, tau - f / f1 - 10.f * slack), hi);
    const float th = tau - 2.f * f * f1 / (2.f * f1 * f1 - f * f2);  // H_f, Eq. 5
    bool take = th >= lo - slack && th <= hi + slack;
    if (!newton_bound && fabsf(f) > 0.5f * f_prev) take = false;
    f_prev = fabsf(f);
    tau = take ? fminf(fmaxf(th, lo), hi) : 0.5f * (lo + hi);
  }
  return tau;
}

// PF (rows of more than 4096 elements, a multiple of 8): persistent
// workgroups, workgroup b taking rows b, b + gridDim.x, ...; the next row's
// values are loaded into registers while the current row iterates, so that
// a workgroup's loads overlap its own iterations (8192 x 8192: 0.108
// against 0.111 ms in fp32, 0.082 against 0.087 ms in bf16; 4096 x 32768
// fp32: 0.235 against 0.269 ms).  Otherwise one workgroup per row: for
// shorter rows the prefetch registers cost occupancy and the persistent
// loop was slower (65536 x 1024: 0.253 against 0.229 ms).  (The backward,
// one reduction per row, got slower the same way: 0.175 against 0.139 ms at
// 8192 x 8192.)
template <typename E, int VPT, int GK, bool PF>
__global__ __launch_bounds__(ROW_NT) void rows_fwd_kernel(RowsArgs a) {
  __shared__ float sh[4 * (ROW_NT / 64)];
  const int n = a.n;
  const float c = a.c, g = a.gamma;
  const E* S = static_cast<const E*>(a.s);
  // Algorithm 1 on row `row`, whose scaled scores are x; writes p and tau.
  auto solve_row = [&](size_t row, float (&x)[VPT]) {
    const float tau = row_tau<VPT, GK>(x, n, a, WgRed<PF>{sh});
    float pv[VPT];
#pragma unroll
    for (int v = 0; v < VPT; ++v) pv[v] = Gamma<GK>::p_only(__builtin_amdgcn_fmed3f(x[v] - tau, 0.f, 1.f), g);
    store_row<VPT>(a.p + row * n, n, pv);
    if (threadIdx.x == 0) a.tau[row] = tau;
  };
  if constexpr (PF) {
    RawRow<E, VPT> nx;
    size_t row = blockIdx.x;
    if ((int64_t)row < a.rows) nx.load(S + row * n, n);
    for (; (int64_t)row < a.rows; row += gridDim.x) {
      float x[VPT];
      nx.scale(n, c, x);
      const size_t next = row + gridDim.x;
      if ((int64_t)next < a.rows) nx.load(S + next * n, n);
      solve_row(row, x);
    }
  } else {
    float x[VPT];
    load_row<E, VPT>(S + (size_t)blockIdx.x * n, n, c, x);
    solve_row(blockIdx.x, x);
  }
}

// Rows of up to 2048 elements: one wave per row, four rows per workgroup,
// reductions by lane exchanges alone (no barriers), so that a workgroup's
// rows do not wait for each other (65536 x 1024 fp32: 0.102 against 0.230
// ms with a workgroup per row; tau differs from that kernel's in the last
// bits, its sums being added in another order).
template <typename E, int VPT, int GK>
__global__ __launch_bounds__(ROW_NT) void rows_fwd_wave_kernel(RowsArgs a) {
  const int64_t row = (int64_t)blockIdx.x * (ROW_NT / 64) + wave_id();
  if (row >= a.rows) return;  // whole waves: the kernel has no barrier
  const int n = a.n, t = lane_id();
  float x[VPT];
  load_row<E, VPT, 64>(static_cast<const E*>(a.s) + (size_t)row * n, n, a.c, x, t);
  const float tau = row_tau<VPT, GK>(x, n, a, WaveRed{});
  float pv[VPT];
#pragma unroll
  for (int v = 0; v < VPT; ++v) pv[v] = Gamma<GK>::p_only(__builtin_amdgcn_fmed3f(x[v] - tau, 0.f, 1.f), a.gamma);
  store_row<VPT, 64>(a.p + (size_t)row * n, n, pv, t);
  if (t == 0) a.tau[row] = tau;
}

// NT threads per row: 256, or 512 and 1024 for rows of more than 8192
// elements, so that a thread holds at most 32 of them (4096 x 32768 fp32:
// 0.288 against 0.475 ms with 256 threads, whose 128 elements each took 256
// registers and left one wave per SIMD).
template <typename E, int VPT, int GK, int NT>
__global__ __launch_bounds__(NT) void rows_bwd_kernel(RowsArgs a) {
  __shared__ float sh[4 * (NT / 64)];
  const size_t row = blockIdx.x;
  const int n = a.n;
  const float c = a.c, g = a.gamma;
  const float tau = a.tau[row];
  float x[VPT];
  load_row<E, VPT, NT>(static_cast<const E*>(a.s) + row * n, n, c, x);
  float u[VPT], gv[VPT];
  load_row<float, VPT, NT>(a.dp + row * n, n, 1.f, gv);  // padding reads -inf; its u is 0
  Sums t{0.f, 0.f, 0.f, 0};
#pragma unroll
  for (int v = 0; v < VPT; ++v) {
    float p;
    Gamma<GK>::pu(__builtin_amdgcn_fmed3f(x[v] - tau, 0.f, 1.f), g, p, u[v]);
    if (u[v] == 0.f) gv[v] = 0.f;
    t.a += u[v];
    t.b = fmaf(u[v], gv[v], t.b);
  }
  const Sums tot = wg_sum<false, NT>(t, sh);
  const float mean = tot.a > 0.f ? tot.b / tot.a : 0.f;  // <u, dp> / sum u
#pragma unroll
  for (int v = 0; v < VPT; ++v) gv[v] = a.scale * u[v] * (gv[v] - mean);
  store_row<VPT, NT>(a.ds + row * n, n, gv);
}

template <typename E, int VPT, int NT>
hipError_t launch_rows_bwd_nt(const RowsArgs& a, hipStream_t s) {
  dim3 grid((unsigned)a.rows), block(NT);
  auto kernel = rows_bwd_kernel<E, VPT, 0, NT>;
  if (a.gk == 1) kernel = rows_bwd_kernel<E, VPT, 1, NT>;
  if (a.gk == 2) kernel = rows_bwd_kernel<E, VPT, 2, NT>;
  if (a.gk == 4) kernel = rows_bwd_kernel<E, VPT, 4, NT>;
  return launch_kernel(kernel, grid, block, s, a);
}

template <typename E, int VPT, bool BWD>
hipError_t launch_rows_v(const RowsArgs& a, hipStream_t s) {
  dim3 grid((unsigned)a.rows), block(ROW_NT);
  if constexpr (BWD) {
    return launch_rows_bwd_nt<E, VPT, ROW_NT>(a, s);
  } else if (VPT < 32 || a.n % 8 != 0) {
    auto kernel = rows_fwd_kernel<E, VPT, 0, false>;
    if (a.gk == 1) kernel = rows_fwd_kernel<E, VPT, 1, false>;
    if (a.gk == 2) kernel = rows_fwd_kernel<E, VPT, 2, false>;
    if (a.gk == 4) kernel = rows_fwd_kernel<E, VPT, 4, false>;
    return launch_kernel(kernel, grid, block, s, a);
  } else {
    auto kernel = rows_fwd_kernel<E, VPT, 0, true>;
    if (a.gk == 1) kernel = rows_fwd_kernel<E, VPT, 1, true>;
    if (a.gk == 2) kernel = rows_fwd_kernel<E, VPT, 2, true>;
    if (a.gk == 4) kernel = rows_fwd_kernel<E, VPT, 4, true>;
    {
      // persistent: as many workgroups as fit on the device at once (at
      // most one per row)
      int dev = 0, cus = 0, per_cu = 0;
      hipError_t e = hipGetDevice(&dev);
      if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
      if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kernel), ROW_NT, 0);
      if (e != hipSuccess) return e;
      const int64_t resident = (int64_t)cus * (per_cu > 0 ? per_cu : 1);
      grid.x = (unsigned)(a.rows < resident ? a.rows : resident);
    }
    return launch_kernel(kernel, grid, block, s, a);
  }
}

template <typename E, int VPT>
hipError_t launch_rows_wave(const RowsArgs& a, hipStream_t s) {
  dim3 grid((unsigned)((a.rows + ROW_NT / 64 - 1) / (ROW_NT / 64))), block(ROW_NT);
  auto kernel = rows_fwd_wave_kernel<E, VPT, 0>;
  if (a.gk == 1) kernel = rows_fwd_wave_kernel<E, VPT, 1>;
  if (a.gk == 2) kernel = rows_fwd_wave_kernel<E, VPT, 2>;
  if (a.gk == 4) kernel = rows_fwd_wave_kernel<E, VPT, 4>;
  return launch_kernel(kernel, grid, block, s, a);
}

// The smallest register row that holds n elements: a wave's for forward
// rows of up to 2048 elements, a wider workgroup's for backward rows of
// more than 8192, else a workgroup of 256 threads'.
template <typename E, bool BWD>
hipError_t launch_rows_e(const RowsArgs& a, hipStream_t s) {
  if (!BWD) {
    if (a.n <= 64 * 4) return launch_rows_wave<E, 4>(a, s);
    if (a.n <= 64 * 16) return launch_rows_wave<E, 16>(a, s);
    if (a.n <= 64 * 32) return launch_rows_wave<E, 32>(a, s);
  } else if (a.n > ROW_NT * 32) {
    if (a.n <= 512 * 32) return launch_rows_bwd_nt<E, 32, 512>(a, s);
    return launch_rows_bwd_nt<E, 32, 1024>(a, s);
  }
  if (a.n <= ROW_NT * 4) return launch_rows_v<E, 4, BWD>(a, s);
  if (a.n <= ROW_NT * 16) return launch_rows_v<E, 16, BWD>(a, s);
  if (a.n <= ROW_NT * 32) return launch_rows_v<E, 32, BWD>(a, s);
  if (a.n <= ROW_NT * 64) return launch_rows_v<E, 64, BWD>(a, s);
  return launch_rows_v<E, 128, BWD>(a, s);
}

}  // namespace

hipError_t launch_rows_fwd(const RowsArgs& a, int dtype, hipStream_t s) {
  return dtype == 0 ? launch_rows_e<__bf16, false>(a, s) : launch_rows_e<float, false>(a, s);
}

hipError_t launch_rows_bwd(const RowsArgs& a, int dtype, hipStream_t s) {
  return dtype == 0 ? launch_rows_e<__bf16, true>(a, s) : launch_rows_e<float, true>(a, s);
}

}  // namespace ea
