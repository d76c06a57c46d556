// ea_fwd.hip -- the sparse alpha-entmax forward, and the column tables.
//
// Tables (Sec. 3.2.1, "pointer-increment lookup tables"; App. A.5): from the
// block mask M, Q_i = {j : M_ij = 1} for every query block i and
// K_j = {i : M_ij = 1} for every key block j, each list ascending, stored as
// a count per block plus a fixed-stride index row of T entries.  The solver
// writes Q_i with its mask row; K_j needs every row of the mask, so extra
// workgroups of the forward's launch build it (the backward reads it).
//
// Forward (Algorithm 2 with the masked loop of App. A.5): for every query
// block i and every key block j in Q_i, recompute S = Q_i K_j^T, P =
// [(alpha-1) S - tau]_+^gamma (Eq. 2) and accumulate O_i += P V_j.  When a
// backward will follow, also accumulate U V_j and sum U with
// U = [(alpha-1) S - tau]_+^(gamma-1) on the support, and write
// O2_i = U V / sum U (the O^(2) of App. A.2).  O is not renormalised: the
// row sums are 1 + f(tau) of the returned tau (Algorithm 1 output).
//
// Precision: S is a bf16 x bf16 product accumulated in fp32; P and U enter
// their products with V as two-term bf16 splits (hi + lo, ~16 significant
// bits), so the only rounding of O beyond fp32 accumulation is its final
// rounding to the input dtype.  With P rounded once to bf16, a row whose
// probability sits on one key (p ~ 1, |v| ~ 5) would carry 2^-9 |v| ~ 0.01
// of operand error on top of the 0.0156 that rounding O ~ 5 to bf16 costs.
//
// gfx950 layout: one workgroup = 4 waves = one 64-row query block; each wave
// holds 32 query rows as MFMA B operands and takes one 32-key half of every
// listed key block, computes S^T (keys x queries) so the probabilities come
// out with one query per lane, and feeds them back as the A operand of P V
// with a permuted contraction order (see ea_common.h).  K and V blocks are
// copied into double-buffered LDS tiles by global_load_lds (the next listed
// block in flight while the current one is consumed); V's operand fragments
// come out of its row-major tile through transposing LDS reads.
#include <type_traits>

#include "ea_common.h"
#include "ea_internal.h"

namespace ea {

namespace {

// --------------------------------------------------------------- tables

// K_j of key block `col` (= bh * T + j), one wave: a ballot and a prefix
// count per 64 query blocks of the mask's column j.
__device__ void column_table(const FwdArgs& a, int col) {
  const int lane = lane_id(), T = a.T;
  const int bh = col / T, j = col % T;
  const uint8_t* M = a.mask + (size_t)bh * T * T;
  int32_t* const out = a.k_index + (size_t)col * T;
  int listed = 0;
  for (int i0 = 0; i0 < T; i0 += 64) {
    const int i = i0 + lane;
    const bool b = i < T && M[(size_t)i * T + j] != 0;
    const unsigned long long m = __ballot(b);
    if (b) out[listed + __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u))] = i;
    listed += __popcll(m);
  }
  if (lane == 0) a.k_count[col] = listed;
}

// --------------------------------------------------------------- forward

constexpr int FWD_NT = 256;
constexpr int FWD_COLS_PER_WG = FWD_NT / 64;  // column tables per extra workgroup

// One 64-row query block per workgroup of 4 waves: wave w takes query half
// qh = w % 2 and, of every listed key block, key half kh = w / 2.  Each wave
// accumulates partial O (and U V, sum U) over its key halves; the two
// partials of a query half are summed through LDS at the end.  The smaller
// per-wave state lets two waves share each SIMD.
//
// Workgroups past the BH * T query blocks build the column tables instead,
// one key block per wave (they come last in the grid).
//
// The bf16 d = 64 inference instances fit 128 registers, so four waves share
// each SIMD instead of three (B8 H12 n1024: 0.049 against 0.052 ms).
template <typename E, int D, int GK, bool TRAIN>
__global__ __launch_bounds__(FWD_NT, !TRAIN && D == 64 && sizeof(E) == 2 ? 4 : 2) void fwd_kernel(FwdArgs a) {
  const int nqb = a.BH * a.T;
  if ((int)blockIdx.x >= nqb) {
    const int col = ((int)blockIdx.x - nqb) * FWD_COLS_PER_WG + wave_id();
    if (col < nqb) column_table(a, col);
    return;
  }
  using TL = Tile<E, D>;
  using M = Mma<E>;
  constexpr int KS = D / M::KW;
  constexpr int NTD = D / 32;
  constexpr int PS = perm_steps<E>();
  __shared__ __attribute__((aligned(16))) E kbuf[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) E vbuf[2][TL::ELEMS];
  __shared__ float usum_x[2][64];
  static_assert(2 * NTD * 16 * 64 * sizeof(float) <= sizeof(kbuf), "partial exchange must fit kbuf");

  const int lane = lane_id(), w = wave_id();
  const int qh = w & 1, kh = w >> 1;
  const int n = a.n, T = a.T;
  const int bh = blockIdx.x % a.BH;
  int qb = blockIdx.x / a.BH;
  if (a.causal) qb = T - 1 - qb;  // longest lists first
  const int q0 = qb * BLK + 32 * qh;
  const int i = q0 + (lane & 31);
  const bool wave_ok = q0 < n;
  const int wave_last = min(n - 1, q0 + 31);
  const size_t head = (size_t)bh * n * D;
  const E* Q = static_cast<const E*>(a.q) + head;
  const E* K = static_cast<const E*>(a.k) + head;
  const E* V = static_cast<const E*>(a.v) + head;
  const float tau = i < n ? a.tau[(size_t)bh * n + i] : 0.f;
  const float c = a.c, g = a.gamma;
  constexpr bool PRECISE = precise_path<E, GK>();
  // fp32 inputs, general alpha: fp64 z near the support edge (ea_common.h)
  [[maybe_unused]] const double tau64 =
      (double)tau + (PRECISE && a.tau_lo && i < n ? (double)a.tau_lo[(size_t)bh * n + i] : 0.0);
  [[maybe_unused]] const float band = PRECISE_BAND * fmaxf(1.f, fabsf(tau));

  typename M::frag qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) qf[kk] = load_row_frag_global<E, D>(Q, i, n, kk);

  // A wave raises its issue priority over its MFMA chains, so that the two
  // waves of a SIMD drift apart (one in its MFMAs while the other maps
  // scores to P and U) instead of contending in the same phase.  At d = 64
  // over S and P V: the kernel took 0.070 against 0.082 ms on B8 H12 n1024,
  // 0.220 against 0.252 on B4 H12 n4096 causal and 0.291 against 0.318 on
  // B1 H8 n16384 causal.  At d = 128 over P V only: 1.017 against 1.027 ms
  // on B1 H16 n8192 at c = 1, 0.580 against 0.604 at c = 16 (over both
  // products it changed nothing there).  Measured for alpha = 1.5 (gamma =
  // 2) only: at alpha = 1.25 (gamma = 4, more work per score between the
  // products) the d = 128 kernel got slower (1.38 against 1.29 ms at c = 1)
  // and at alpha = 2 it made no difference, so the other exponents do
  // without, as do the dK/dV kernels (1.31 against 1.27 ms at d = 128).
  constexpr bool PRIO_PV = GK == 2;
  constexpr bool PRIO_S = PRIO_PV && D == 64;

  const int32_t* list = a.q_index + ((size_t)bh * T + qb) * T;
  const int cnt = a.q_count[(size_t)bh * T + qb];

  f32x16 o[NTD], o2[NTD];
#pragma unroll
  for (int t = 0; t < NTD; ++t) {
    o[t] = zero16();
    if constexpr (TRAIN) o2[t] = zero16();
  }
  float usum = 0.f;

  // 0 = no valid key for this wave, 1 = all valid, 2 = per-element masking
  auto sub_kind = [&](int j0) {
    if (!wave_ok || j0 >= n || (a.causal && j0 > wave_last)) return 0;
    if (j0 + 31 >= n || (a.causal && j0 + 31 > q0)) return 2;
    return 1;
  };

  DmaPlan<E, D, FWD_NT> dma;
  dma.init();
  auto issue = [&](int e) {
    const int kb = list[e];
    dma.issue(kbuf[e & 1], K, kb * BLK, n);
    dma.issue(vbuf[e & 1], V, kb * BLK, n);
  };
  if (cnt > 0) issue(0);
  for (int e = 0; e < cnt; ++e) {
    dma_wait();
    __syncthreads();
    if (e + 1 < cnt) issue(e + 1);
    const E* kt = kbuf[e & 1];
    const E* vt = vbuf[e & 1];
    const int j0 = list[e] * BLK + 32 * kh;
    const int kind = sub_kind(j0);
    if (kind == 0) continue;
    // S^T = K Q^T for this wave's 32 keys x 32 queries
    f32x16 s = zero16();
    if constexpr (PRIO_S) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) s = M::mma(lds_row_frag<E, D>(kt, 32 * kh + (lane & 31), kk), qf[kk], s);
    if constexpr (PRIO_S) __builtin_amdgcn_s_setprio(0);
    if (kind == 2) {  // invalid keys -> -inf, so [x - tau]_+ is exactly 0 there
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = j0 + crow(r);
        if (!(j < n && (!a.causal || j <= i))) s[r] = -INFINITY;
      }
    }
    if constexpr (GK == 4 && !PRECISE) {
      // Maps and contracts one step's elements at a time, so that fewer
      // values are live: at alpha = 1.25 (gamma = 4) the training instance
      // at d = 128 spilled 48 bytes per lane with all sixteen mapped first,
      // and ran 1.18 against 1.29 ms this way (B1 H16 n8192, c = 1).  For the
      // other exponents the sixteen mapped first were faster (alpha = 1.5:
      // 1.034 against 1.057 ms).
      constexpr int EPS = 16 / PS;  // elements per contraction step
#pragma unroll
      for (int t = 0; t < PS; ++t) {
        float pt[16], ut[16];
#pragma unroll
        for (int e = 0; e < EPS; ++e) {
          const float zp = relu_z(c, s[EPS * t + e], tau);
          if constexpr (TRAIN) {
            Gamma<GK>::pu(zp, g, pt[EPS * t + e], ut[EPS * t + e]);
            usum += ut[EPS * t + e];
          } else {
            pt[EPS * t + e] = Gamma<GK>::p_only(zp, g);
          }
        }
        typename M::frag ph, pl, uh, ul;
        M::pack_split(pt, t, ph, pl);
        if constexpr (TRAIN) M::pack_split(ut, t, uh, ul);
#pragma unroll
        for (int nt = 0; nt < NTD; ++nt) {
          const typename M::frag vb = lds_perm_frag<E, D>(vt, 32 * nt, 32 * kh, t);
          o[nt] = M::mma(ph, vb, o[nt]);
          if constexpr (!M::exact_operands) o[nt] = M::mma(pl, vb, o[nt]);
          if constexpr (TRAIN) {
            o2[nt] = M::mma(uh, vb, o2[nt]);
            if constexpr (!M::exact_operands) o2[nt] = M::mma(ul, vb, o2[nt]);
          }
        }
      }
      continue;
    }
    float p[16], u[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float zp;
      if constexpr (PRECISE) {
        zp = precise_relu_z<D>(i < n, c, s[r], tau, band, tau64,
                               reinterpret_cast<const float*>(Q) + (size_t)i * D,
                               reinterpret_cast<const float*>(K) + (size_t)(j0 + crow(r)) * D, a.c64);
      } else {
        zp = relu_z(c, s[r], tau);
      }
      if constexpr (TRAIN) {
        Gamma<GK>::pu(zp, g, p[r], u[r]);
        usum += u[r];
      } else {
        p[r] = Gamma<GK>::p_only(zp, g);
      }
    }
    if constexpr (PRIO_PV) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int t = 0; t < PS; ++t) {
      typename M::frag ph, pl, uh, ul;
      M::pack_split(p, t, ph, pl);
      if constexpr (TRAIN) M::pack_split(u, t, uh, ul);
#pragma unroll
      for (int nt = 0; nt < NTD; ++nt) {
        const typename M::frag vb = lds_perm_frag<E, D>(vt, 32 * nt, 32 * kh, t);
        o[nt] = M::mma(ph, vb, o[nt]);
        if constexpr (!M::exact_operands) o[nt] = M::mma(pl, vb, o[nt]);
        if constexpr (TRAIN) {
          o2[nt] = M::mma(uh, vb, o2[nt]);
          if constexpr (!M::exact_operands) o2[nt] = M::mma(ul, vb, o2[nt]);
        }
      }
    }
    if constexpr (PRIO_PV) __builtin_amdgcn_s_setprio(0);
  }

  // Sum the two key-half partials of each query half through LDS: first O
  // and sum U, then O2; kh = 1 hands over, kh = 0 adds and writes.
  if constexpr (TRAIN) usum += __shfl_xor(usum, 32);
  float* xch = reinterpret_cast<float*>(&kbuf[0][0]);
  auto xidx = [&](int nt, int r) { return ((qh * NTD + nt) * 16 + r) * 64 + lane; };
  __syncthreads();
  if (kh == 1) {
#pragma unroll
    for (int nt = 0; nt < NTD; ++nt)
#pragma unroll
      for (int r = 0; r < 16; ++r) xch[xidx(nt, r)] = o[nt][r];
    if (lane < 32) usum_x[qh][lane] = usum;
  }
  __syncthreads();
  if (kh == 0) {
#pragma unroll
    for (int nt = 0; nt < NTD; ++nt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[nt][r] += xch[xidx(nt, r)];
    if constexpr (TRAIN) usum += usum_x[qh][lane & 31];
  }
  if constexpr (TRAIN) {
    __syncthreads();
    if (kh == 1) {
#pragma unroll
      for (int nt = 0; nt < NTD; ++nt)
#pragma unroll
        for (int r = 0; r < 16; ++r) xch[xidx(nt, r)] = o2[nt][r];
    }
    __syncthreads();
    if (kh == 0) {
#pragma unroll
      for (int nt = 0; nt < NTD; ++nt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o2[nt][r] += xch[xidx(nt, r)];
    }
  }
  if (kh == 1 || !wave_ok) return;

  E* O = static_cast<E*>(a.o) + head;
  float* O2 = a.o2 + head;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = crow(r);
    const int ir = q0 + row;
    float us = 0.f;
    if constexpr (TRAIN) us = __shfl(usum, row);
    if (ir < n) {
#pragma unroll
      for (int nt = 0; nt < NTD; ++nt) {
        const size_t off = (size_t)ir * D + 32 * nt + (lane & 31);
        O[off] = (E)o[nt][r];
        if constexpr (TRAIN) O2[off] = us > 0.f ? o2[nt][r] / us : 0.f;
      }
    }
  }
}

// The column tables serve the backward only, so an inference forward
// (TRAIN false) launches no workgroups for them.
template <typename E, int D, bool TRAIN>
hipError_t launch_fwd_dt(const FwdArgs& a, hipStream_t s) {
  const int nqb = a.BH * a.T;
  const int ncol = TRAIN ? (nqb + FWD_COLS_PER_WG - 1) / FWD_COLS_PER_WG : 0;
  dim3 grid((unsigned)(nqb + ncol)), block(FWD_NT);
  auto kernel = fwd_kernel<E, D, 0, TRAIN>;
  if (a.gk == 1) kernel = fwd_kernel<E, D, 1, TRAIN>;
  if (a.gk == 2) kernel = fwd_kernel<E, D, 2, TRAIN>;
  if (a.gk == 4) kernel = fwd_kernel<E, D, 4, TRAIN>;
  return launch_kernel(kernel, grid, block, s, a);
}

template <typename E, int D>
hipError_t launch_fwd_d(const FwdArgs& a, bool train, hipStream_t s) {
  return train ? launch_fwd_dt<E, D, true>(a, s) : launch_fwd_dt<E, D, false>(a, s);
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a, int dtype, int head_dim, bool train, hipStream_t s) {
  if (dtype == 0)
    return head_dim == 64 ? launch_fwd_d<__bf16, 64>(a, train, s) : launch_fwd_d<__bf16, 128>(a, train, s);
  return head_dim == 64 ? launch_fwd_d<float, 64>(a, train, s) : launch_fwd_d<float, 128>(a, train, s);
}

}  // namespace ea
