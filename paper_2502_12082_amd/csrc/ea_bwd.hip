// ea_bwd.hip -- sparse alpha-entmax attention backward.
//
// With tau from the forward, u_ij = [x_ij - tau_i]_+^(gamma-1) on the support
// (= p^(2-alpha), the sparse Jacobian Diag(u) - u u^T / |u|_1 of Sec. 3.2.2)
// and O2 saved by the forward (App. A.2):
//   delta_i = <dO_i, O2_i>                                   (App. A.2)
//   dP_ij   = <dO_i, v_j>,  dS_ij = u_ij (dP_ij - delta_i)    (App. A.2)
//   dV_j = sum_{i in K_j} P_ij^T dO_i                         (Eq. 13)
//   dK_j = scale * sum_{i in K_j} dS_ij^T q_i                 (Eq. 12)
//   dQ_i = scale * sum_{j in Q_i} dS_ij k_j                   (Eq. 11)
// split into a delta pre-kernel, a dK/dV kernel over key blocks and a dQ
// kernel over query blocks (Algorithms 4 and 5, visiting only the blocks of
// the lookup tables as in App. A.5).  `scale` appears because the entmax
// input is scale * Q K^T; no alpha factor survives the chain rule.
//
// Precision: S and dP are bf16 x bf16 products accumulated in fp32; P is
// rounded to bf16 for P^T dO; dS is fed to the MFMA as a two-term bf16 split
// (hi + lo) so dK and dQ keep ~16 mantissa bits of dS; outputs are fp32.
//
// gfx950 layout: 32 resident rows per wave in registers (K and V rows for
// dK/dV; Q and dO rows for dQ); the other side's 64-row tiles are copied by
// global_load_lds into row-major LDS tiles (two stages; three in the bf16
// d = 128 dK/dV kernel), read directly for S and dP and through transposing
// LDS reads for the permuted contractions P^T dO, dS^T Q and dS K.  The dK/dV
// work has two forms: dkdv_kernel (2 waves per key block, every column) and,
// for bf16 at d = 128, dkdv2_kernel (8 waves over two key blocks, each wave
// half of the columns, S and dP operands shared through LDS).  No atomics:
// every output row has one owner, so results are deterministic.
#include <type_traits>

#include "ea_common.h"
#include "ea_internal.h"

namespace ea {

namespace {

constexpr int BWD_NT = 128;

// ------------------------------------------------------------------ delta

template <typename E, int D>
__global__ __launch_bounds__(256) void delta_kernel(DeltaArgs a) {
  constexpr int PER = D / 16;  // 16 lanes per row
  const long long row = (long long)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int sl = threadIdx.x & 15;
  float acc = 0.f;
  if (row < a.rows) {
    const E* dO = static_cast<const E*>(a.dout) + row * D + sl * PER;
    const float* o2 = a.o2 + row * D + sl * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc = fmaf((float)dO[e], o2[e], acc);
  }
#pragma unroll
  for (int m = 8; m >= 1; m >>= 1) acc += __shfl_xor(acc, m);
  if (row < a.rows && sl == 0) a.delta[row] = acc;
}

// ------------------------------------------------------------------ dK dV

template <typename E, int D, int GK>
__global__ __launch_bounds__(BWD_NT) void dkdv_kernel(BwdArgs a) {
  using TL = Tile<E, D>;
  using M = Mma<E>;
  constexpr int KS = D / M::KW;
  constexpr int NTD = D / 32;
  constexpr int PS = perm_steps<E>();
  __shared__ __attribute__((aligned(16))) E qbuf[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) E dobuf[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) float tau_s[2][BLK];
  __shared__ __attribute__((aligned(16))) float del_s[2][BLK];

  const int lane = lane_id(), w = wave_id();
  const int n = a.n, T = a.T;
  const int bh = blockIdx.x % a.BH;
  const int kb = blockIdx.x / a.BH;  // causal: small kb has the longest list
  const int k0 = kb * BLK + 32 * w;
  const int j = k0 + (lane & 31);
  const bool wave_ok = k0 < n;
  const size_t head = (size_t)bh * n * D;
  const E* Qg = static_cast<const E*>(a.q) + head;
  const E* Kg = static_cast<const E*>(a.k) + head;
  const E* Vg = static_cast<const E*>(a.v) + head;
  const E* dOg = static_cast<const E*>(a.dout) + head;
  const float* taug = a.tau + (size_t)bh * n;
  const float* delg = a.delta + (size_t)bh * n;
  const float c = a.c, g = a.gamma;
  constexpr bool PRECISE = precise_path<E, GK>();

  typename M::frag kf[KS], vf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    kf[kk] = load_row_frag_global<E, D>(Kg, j, n, kk);
    vf[kk] = load_row_frag_global<E, D>(Vg, j, n, kk);
  }

  // Without tables (the no-mask mode) every valid query block is visited.
  const bool dense = a.k_index == nullptr;
  const int32_t* list = dense ? nullptr : a.k_index + ((size_t)bh * T + kb) * T;
  const int cnt = dense ? (a.causal ? T - kb : T) : a.k_count[(size_t)bh * T + kb];
  auto qb_of = [&](int e) { return dense ? (a.causal ? kb + e : e) : list[e]; };

  f32x16 dk[NTD], dv[NTD];
#pragma unroll
  for (int t = 0; t < NTD; ++t) {
    dk[t] = zero16();
    dv[t] = zero16();
  }

  // One 32-query half of the staged block against this wave's 32 keys:
  // S = Q K^T, dP = dO V^T (rows = queries), then dV += P^T dO, dK += dS^T Q.
  // Masked sub-tiles set invalid scores to -inf first (the clamp of
  // [x - tau]_+ then gives exactly 0), so one code path updates dK and dV.
  auto block = [&](bool masked, const E* qt, const E* dt, const float* ts, const float* ds_,
                   int qh, int i0) {
    f32x16 s = zero16(), dp = zero16();
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      s = M::mma(lds_row_frag<E, D>(qt, 32 * qh + (lane & 31), kk), kf[kk], s);
      dp = M::mma(lds_row_frag<E, D>(dt, 32 * qh + (lane & 31), kk), vf[kk], dp);
    }
    if (masked) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = i0 + crow(r);
        if (!(i < n && j < n && (!a.causal || j <= i))) s[r] = -INFINITY;
      }
    }
    float p[16], dsv[16];
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      // rows 8 g4 + 4h + (0..3) of this half: one 16-byte read each for tau, delta
      const int q4 = 32 * qh + 8 * g4 + 4 * (lane >> 5);
      const f32x4 tq = *reinterpret_cast<const f32x4*>(ts + q4);
      const f32x4 dq4 = *reinterpret_cast<const f32x4*>(ds_ + q4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * g4 + e;
        float zp;
        if constexpr (PRECISE) {
          // fp64 z near the support edge (ea_common.h); invalid pairs hold -inf
          const int i = i0 + crow(r);
          const bool ok = i < n && j < n;
          const float band = PRECISE_BAND * fmaxf(1.f, fabsf(tq[e]));
          const float raw = fmaf(c, s[r], -tq[e]);
          double t64 = tq[e];
          if (ok && fabsf(raw) < band && a.tau_lo) t64 += (double)a.tau_lo[(size_t)bh * n + i];
          zp = precise_relu_z<D>(ok, c, s[r], tq[e], band, t64,
                                 reinterpret_cast<const float*>(Qg) + (size_t)i * D,
                                 reinterpret_cast<const float*>(Kg) + (size_t)j * D, a.c64);
        } else {
          zp = relu_z(c, s[r], tq[e]);
        }
        float u;
        Gamma<GK>::pu(zp, g, p[r], u);
        dsv[r] = u * (dp[r] - dq4[e]);
      }
    }
#pragma unroll
    for (int t = 0; t < PS; ++t) {
      const typename M::frag pa = M::pack(p, t);
      typename M::frag dh, dl;
      M::pack_split(dsv, t, dh, dl);
#pragma unroll
      for (int nt = 0; nt < NTD; ++nt) {
        dv[nt] = M::mma(pa, lds_perm_frag<E, D>(dt, 32 * nt, 32 * qh, t), dv[nt]);
        const typename M::frag qb_ = lds_perm_frag<E, D>(qt, 32 * nt, 32 * qh, t);
        dk[nt] = M::mma(dh, qb_, dk[nt]);
        if constexpr (!M::exact_operands) dk[nt] = M::mma(dl, qb_, dk[nt]);
      }
    }
  };

  float tv = 0.f, dlv = 0.f;
  DmaPlan<E, D, BWD_NT> dma;
  dma.init();
  auto issue = [&](int e) {
    const int qb = qb_of(e);
    dma.issue(qbuf[e & 1], Qg, qb * BLK, n);
    dma.issue(dobuf[e & 1], dOg, qb * BLK, n);
    if (threadIdx.x < BLK) {
      const int r = min(qb * BLK + (int)threadIdx.x, n - 1);
      tv = taug[r];
      dlv = delg[r];
    }
  };
  if (cnt > 0) issue(0);
  for (int e = 0; e < cnt; ++e) {
    dma_wait();
    if (threadIdx.x < BLK) {
      tau_s[e & 1][threadIdx.x] = tv;
      del_s[e & 1][threadIdx.x] = dlv;
    }
    __syncthreads();
    const int qb = qb_of(e);
    if (e + 1 < cnt) issue(e + 1);
    if (!wave_ok) continue;
    const E* qt = qbuf[e & 1];
    const E* dt = dobuf[e & 1];
#pragma unroll
    for (int qh = 0; qh < 2; ++qh) {
      const int i0 = qb * BLK + 32 * qh;
      if (i0 >= n || (a.causal && k0 > i0 + 31)) continue;
      const bool masked = i0 + 31 >= n || k0 + 31 >= n || (a.causal && k0 + 31 > i0);
      block(masked, qt, dt, tau_s[e & 1], del_s[e & 1], qh, i0);
    }
  }

  if (!wave_ok) return;
  float* dK = a.dk + head;
  float* dV = a.dv + head;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int key = k0 + crow(r);
    if (key < n) {
#pragma unroll
      for (int nt = 0; nt < NTD; ++nt) {
        const size_t off = (size_t)key * D + 32 * nt + (lane & 31);
        dK[off] = a.scale * dk[nt][r];
        dV[off] = dv[nt][r];
      }
    }
  }
}

// ------------------------------------------------------- dK dV, bf16 inputs

// Eight waves over two adjacent key blocks (2m and 2m + 1).  Wave w owns key
// block 2m + (w >> 2), key half kh = (w >> 1) & 1 (32 keys, as above) and
// column half ch = w & 1 of dK and dV.  For each staged query block the wave
// forms S and dP of its keys against query half ch only, turns them into the
// operands P, dS_hi and dS_lo of the permuted contractions and posts those
// through LDS; its partner (same keys, other column half) posts the other
// query half.  Each wave then accumulates dV and dK for its columns over
// both query halves.  Half the accumulators and no repeated products let
// two waves share each SIMD, while every product is formed once.  The two
// key blocks visit the union of their query-block lists (both ascending);
// the waves of a key block that does not list the staged query block only
// keep the barriers.
//
// The Q and dO tiles (with their tau and delta) go through three LDS stages,
// so each copy has two steps to land, and the barriers wait only for LDS
// traffic: a plain workgroup barrier would also wait for the copies in
// flight.  The tables are read by scalar loads for the same reason.
constexpr int BWD2_NT = 512;

template <int D, int GK>
__global__ __launch_bounds__(BWD2_NT, 2) void dkdv2_kernel(BwdArgs a) {
  using E = __bf16;
  using TL = Tile<E, D>;
  using M = Mma<E>;
  using F = typename M::frag;
  constexpr int KS = D / M::KW;
  constexpr int NTH = D / 64;  // 32-column output tiles per wave
  constexpr int PS = perm_steps<E>();
  // three stages: block e is read while e + 1 and e + 2 are in flight
  __shared__ __attribute__((aligned(16))) E qbuf[3][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) E dobuf[3][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) float tau_s[3][BLK];
  __shared__ __attribute__((aligned(16))) float del_s[3][BLK];
  // operands posted by each wave: [wave][P, dS hi, dS lo][step][lane]
  __shared__ __attribute__((aligned(16))) u32x4 post[BWD2_NT / 64][3][PS][64];

  const int lane = lane_id(), w = wave_id();
  const int kh = (w >> 1) & 1, ch = w & 1;
  const int n = a.n, T = a.T;
  const int bh = blockIdx.x % a.BH;
  const int kbA = 2 * (blockIdx.x / a.BH);  // causal: small key blocks have the longest lists
  const int kbB = kbA + 1;
  const bool mineA = (w >> 2) == 0;
  const int k0 = (mineA ? kbA : kbB) * BLK + 32 * kh;
  const int j = k0 + (lane & 31);
  const bool wave_ok = k0 < n;
  const size_t head = (size_t)bh * n * D;
  const E* Qg = static_cast<const E*>(a.q) + head;
  const E* Kg = static_cast<const E*>(a.k) + head;
  const E* Vg = static_cast<const E*>(a.v) + head;
  const E* dOg = static_cast<const E*>(a.dout) + head;
  [[maybe_unused]] const float* taug = a.tau + (size_t)bh * n;  // read by tile copies
  [[maybe_unused]] const float* delg = a.delta + (size_t)bh * n;
  const float c = a.c, g = a.gamma;

  F kf[KS], vf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    kf[kk] = load_row_frag_global<E, D>(Kg, j, n, kk);
    vf[kk] = load_row_frag_global<E, D>(Vg, j, n, kk);
  }

  // Query-block lists of the two key blocks (without tables, in the no-mask
  // mode, every valid query block), merged in ascending order.
  const bool dense = a.k_index == nullptr;
  // The tables are read through the constant address space (scalar loads),
  // so that reading them does not wait on the tile copies in flight.
  typedef const __attribute__((address_space(4))) int32_t ci32;
  const ci32* kcount = (const ci32*)a.k_count;
  const ci32* kindex = (const ci32*)a.k_index;
  auto count_of = [&](int kb) {
    if (kb >= T) return 0;
    return dense ? (a.causal ? T - kb : T) : kcount[(size_t)bh * T + kb];
  };
  auto entry_of = [&](int kb, int e) {
    return dense ? (a.causal ? kb + e : e) : kindex[((size_t)bh * T + kb) * T + e];
  };
  const int nA = count_of(kbA), nB = count_of(kbB);
  int pA = 0, pB = 0;
  // the next query block of the union, and whether each key block lists it
  auto next = [&](int& qb, bool& inA, bool& inB) {
    const int hA = pA < nA ? entry_of(kbA, pA) : T;
    const int hB = pB < nB ? entry_of(kbB, pB) : T;
    qb = min(hA, hB);
    inA = hA == qb;
    inB = hB == qb;
    pA += inA ? 1 : 0;
    pB += inB ? 1 : 0;
    return qb < T;
  };

  f32x16 dk[NTH], dv[NTH];
#pragma unroll
  for (int t = 0; t < NTH; ++t) {
    dk[t] = zero16();
    dv[t] = zero16();
  }

  // S = Q K^T, dP = dO V^T of query half qh (rows = queries) for this wave's
  // keys; masked sub-tiles set invalid scores to -inf (then P = dS = 0).
  auto operands = [&](const E* qt, const E* dt, const float* ts, const float* ds_, int qh,
                      bool masked, int i0, F* pa, F* dh, F* dl) {
    f32x16 s = zero16(), dp = zero16();
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      s = M::mma(lds_row_frag<E, D>(qt, 32 * qh + (lane & 31), kk), kf[kk], s);
      dp = M::mma(lds_row_frag<E, D>(dt, 32 * qh + (lane & 31), kk), vf[kk], dp);
    }
    if (masked) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = i0 + crow(r);
        if (!(i < n && j < n && (!a.causal || j <= i))) s[r] = -INFINITY;
      }
    }
    float p[16], dsv[16];
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int q4 = 32 * qh + 8 * g4 + 4 * (lane >> 5);
      const f32x4 tq = *reinterpret_cast<const f32x4*>(ts + q4);
      const f32x4 dq4 = *reinterpret_cast<const f32x4*>(ds_ + q4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * g4 + e;
        const float zp = relu_z(c, s[r], tq[e]);
        float u;
        Gamma<GK>::pu(zp, g, p[r], u);
        dsv[r] = u * (dp[r] - dq4[e]);
      }
    }
#pragma unroll
    for (int t = 0; t < PS; ++t) {
      pa[t] = M::pack(p, t);
      M::pack_split(dsv, t, dh[t], dl[t]);
    }
  };
  // dV += P^T dO and dK += dS^T Q over query half qh, this wave's columns
  auto accum = [&](const E* qt, const E* dt, int qh, const F* pa, const F* dh, const F* dl) {
#pragma unroll
    for (int t = 0; t < PS; ++t) {
#pragma unroll
      for (int nt = 0; nt < NTH; ++nt) {
        const int col0 = 32 * (ch * NTH + nt);
        dv[nt] = M::mma(pa[t], lds_perm_frag<E, D>(dt, col0, 32 * qh, t), dv[nt]);
        const F qb_ = lds_perm_frag<E, D>(qt, col0, 32 * qh, t);
        dk[nt] = M::mma(dh[t], qb_, dk[nt]);
        dk[nt] = M::mma(dl[t], qb_, dk[nt]);
      }
    }
  };
  auto half_valid = [&](int i0) { return !(i0 >= n || (a.causal && k0 > i0 + 31)); };
  auto half_masked = [&](int i0) {
    return i0 + 31 >= n || k0 + 31 >= n || (a.causal && k0 + 31 > i0);
  };

  using Plan = DmaPlan<E, D, BWD2_NT>;
  static_assert(Plan::NI % Plan::NW == 0 && 2 * Plan::PER + 2 <= 15, "copy counts");
  Plan dma;
  dma.init();
  // Copies of query block qb into stage b: the Q and dO tiles, and (wave 0)
  // its tau and delta values, all by global_load_lds.
  auto issue = [&](int qb, int b) {
    dma.issue(qbuf[b], Qg, qb * BLK, n);
    dma.issue(dobuf[b], dOg, qb * BLK, n);
#if defined(__HIP_DEVICE_COMPILE__)
    if (w == 0) {
      const int r = min(qb * BLK + lane, n - 1);
      __builtin_amdgcn_global_load_lds(taug + r, to_lds(&tau_s[b][0]), 4, 0, 0);
      __builtin_amdgcn_global_load_lds(delg + r, to_lds(&del_s[b][0]), 4, 0, 0);
    }
#endif
  };
  // Workgroup barrier for LDS traffic only: this wave's LDS operations
  // complete first, but copies still in flight are not waited for (the
  // plain barrier would also wait for every global load, so the next
  // stages' copies would have to land first).
  auto lds_barrier = [&]() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
  // Waits until every copy but those of the latest issue has landed (the
  // counter completes in issue order; wave 0 issues two more per stage).
  auto wait_all_but_latest = [&]() {
    if (w == 0) {
      __builtin_amdgcn_s_waitcnt(0x0F70 | (2 * Plan::PER + 2));
    } else {
      __builtin_amdgcn_s_waitcnt(0x0F70 | (2 * Plan::PER));
    }
  };
  // S, dP, P, dS of query half ch (kept for this wave, posted for its partner)
  F pa[PS], dh[PS], dl[PS];
  auto phase1 = [&](int qb, int b, int tb) {
    const int i0 = qb * BLK + 32 * ch;
    if (!half_valid(i0)) return;
    operands(qbuf[b], dobuf[b], tau_s[tb], del_s[tb], ch, half_masked(i0), i0, pa, dh, dl);
#pragma unroll
    for (int t = 0; t < PS; ++t) {
      post[w][0][t][lane] = __builtin_bit_cast(u32x4, pa[t]);
      post[w][1][t][lane] = __builtin_bit_cast(u32x4, dh[t]);
      post[w][2][t][lane] = __builtin_bit_cast(u32x4, dl[t]);
    }
  };
  // both query halves into this wave's columns: the partner's half first
  auto phase2 = [&](int qb, int b) {
    if (half_valid(qb * BLK + 32 * (ch ^ 1))) {
      F xa[PS], xh[PS], xl[PS];
#pragma unroll
      for (int t = 0; t < PS; ++t) {
        xa[t] = __builtin_bit_cast(F, post[w ^ 1][0][t][lane]);
        xh[t] = __builtin_bit_cast(F, post[w ^ 1][1][t][lane]);
        xl[t] = __builtin_bit_cast(F, post[w ^ 1][2][t][lane]);
      }
      accum(qbuf[b], dobuf[b], ch ^ 1, xa, xh, xl);
    }
    if (half_valid(qb * BLK + 32 * ch)) accum(qbuf[b], dobuf[b], ch, pa, dh, dl);
  };

  // Union entries e (stage b0), e + 1 and e + 2 (in flight).
  int q0 = 0, q1 = 0;
  bool a0 = false, b0_ = false, a1 = false, b1_ = false;
  bool h0 = next(q0, a0, b0_);
  bool h1 = h0 && next(q1, a1, b1_);
  if (h0) issue(q0, 0);
  if (h1) issue(q1, 1);
  int st = 0;
  while (h0) {
    int q2 = 0;
    bool a2 = false, b2_ = false;
    const bool h2 = h1 && next(q2, a2, b2_);
    if (h1) {
      wait_all_but_latest();
    } else {
      dma_wait();
    }
    // block q0 is staged (each wave waited for its own copies); every wave
    // is done with the previous step, whose stage receives block q2
    lds_barrier();
    if (h2) issue(q2, st == 0 ? 2 : st - 1);
    const bool act = wave_ok && (mineA ? a0 : b0_);
    if (act) phase1(q0, st, st);
    lds_barrier();  // the posted operands are visible
    if (act) phase2(q0, st);
    q0 = q1;
    a0 = a1;
    b0_ = b1_;
    h0 = h1;
    q1 = q2;
    a1 = a2;
    b1_ = b2_;
    h1 = h2;
    st = st == 2 ? 0 : st + 1;
  }

  if (!wave_ok) return;
  float* dK = a.dk + head;
  float* dV = a.dv + head;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int key = k0 + crow(r);
    if (key < n) {
#pragma unroll
      for (int nt = 0; nt < NTH; ++nt) {
        const size_t off = (size_t)key * D + 32 * (ch * NTH + nt) + (lane & 31);
        dK[off] = a.scale * dk[nt][r];
        dV[off] = dv[nt][r];
      }
    }
  }
}

// --------------------------------------------------------------------- dQ

constexpr int DQ_NT = 256;

// One 64-row query block per workgroup of 4 waves: wave w takes query half
// qh = w % 2 and, of every listed key block, key half kh = w / 2, so each
// wave holds only its 32 query rows and one partial dQ; the two key-half
// partials are summed through LDS at the end.  Halving the per-wave state
// lets two waves share each SIMD.  At d = 128 a wave raises its issue
// priority over its dQ products, so that the two waves of a SIMD drift
// apart (B1 H16 n8192: 0.905 against 0.922 ms at alpha = 1.5, c = 1, 0.505
// against 0.531 at c = 16, 0.925 against 0.941 at alpha = 1.25, c = 1, 0.806
// against 0.844 at alpha = 2, c = 1); at d = 64 that was slower (0.256
// against 0.252 ms on B1 H8 n16384 causal).
template <typename E, int D, int GK>
__global__ __launch_bounds__(DQ_NT, 2) void dq_kernel(BwdArgs a) {
  using TL = Tile<E, D>;
  using M = Mma<E>;
  constexpr int KS = D / M::KW;
  constexpr int NTD = D / 32;
  constexpr int PS = perm_steps<E>();
  __shared__ __attribute__((aligned(16))) E kbuf[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) E vbuf[2][TL::ELEMS];
  static_assert(2 * NTD * 16 * 64 * sizeof(float) <= sizeof(kbuf), "dQ exchange must fit kbuf");

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
  const E* Qg = static_cast<const E*>(a.q) + head;
  const E* Kg = static_cast<const E*>(a.k) + head;
  const E* Vg = static_cast<const E*>(a.v) + head;
  const E* dOg = static_cast<const E*>(a.dout) + head;
  const float tau = i < n ? a.tau[(size_t)bh * n + i] : 0.f;
  const float del = i < n ? a.delta[(size_t)bh * n + i] : 0.f;
  const float c = a.c, g = a.gamma;
  constexpr bool PRECISE = precise_path<E, GK>();
  // fp32 inputs, general alpha: fp64 z near the support edge (ea_common.h)
  [[maybe_unused]] const double tau64 =
      (double)tau + (PRECISE && a.tau_lo && i < n ? (double)a.tau_lo[(size_t)bh * n + i] : 0.0);
  [[maybe_unused]] const float band = PRECISE_BAND * fmaxf(1.f, fabsf(tau));

  typename M::frag qf[KS], df[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    qf[kk] = load_row_frag_global<E, D>(Qg, i, n, kk);
    df[kk] = load_row_frag_global<E, D>(dOg, i, n, kk);
  }

  // Without tables (the no-mask mode) every valid key block is visited.
  const bool dense = a.q_index == nullptr;
  const int32_t* list = dense ? nullptr : a.q_index + ((size_t)bh * T + qb) * T;
  const int cnt = dense ? (a.causal ? qb + 1 : T) : a.q_count[(size_t)bh * T + qb];
  auto kb_of = [&](int e) { return dense ? e : list[e]; };

  f32x16 dq[NTD];
#pragma unroll
  for (int t = 0; t < NTD; ++t) dq[t] = zero16();

  // 0 = no valid key for this wave, 1 = all valid, 2 = per-element masking
  auto sub_kind = [&](int j0) {
    if (!wave_ok || j0 >= n || (a.causal && j0 > wave_last)) return 0;
    if (j0 + 31 >= n || (a.causal && j0 + 31 > q0)) return 2;
    return 1;
  };

  DmaPlan<E, D, DQ_NT> dma;
  dma.init();
  auto issue = [&](int e) {
    const int kb = kb_of(e);
    dma.issue(kbuf[e & 1], Kg, kb * BLK, n);
    dma.issue(vbuf[e & 1], Vg, kb * BLK, n);
  };
  if (cnt > 0) issue(0);
  for (int e = 0; e < cnt; ++e) {
    dma_wait();
    __syncthreads();
    if (e + 1 < cnt) issue(e + 1);
    const E* kt = kbuf[e & 1];
    const E* vt = vbuf[e & 1];
    const int j0 = kb_of(e) * BLK + 32 * kh;
    const int kind = sub_kind(j0);
    if (kind == 0) continue;
    // S^T = K Q^T and dP^T = V dO^T for this wave's 32 keys x 32 queries
    f32x16 s = zero16(), dp = zero16();
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      s = M::mma(lds_row_frag<E, D>(kt, 32 * kh + (lane & 31), kk), qf[kk], s);
      dp = M::mma(lds_row_frag<E, D>(vt, 32 * kh + (lane & 31), kk), df[kk], dp);
    }
    if (kind == 2) {  // invalid keys -> -inf, so [x - tau]_+ is exactly 0 there
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int jj = j0 + crow(r);
        if (!(jj < n && (!a.causal || jj <= i))) s[r] = -INFINITY;
      }
    }
    float dsv[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float zp;
      if constexpr (PRECISE) {
        zp = precise_relu_z<D>(i < n, c, s[r], tau, band, tau64,
                               reinterpret_cast<const float*>(Qg) + (size_t)i * D,
                               reinterpret_cast<const float*>(Kg) + (size_t)(j0 + crow(r)) * D, a.c64);
      } else {
        zp = relu_z(c, s[r], tau);
      }
      float p, u;
      Gamma<GK>::pu(zp, g, p, u);
      dsv[r] = u * (dp[r] - del);
    }
    if constexpr (D == 128) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int t = 0; t < PS; ++t) {
      typename M::frag dh, dl;
      M::pack_split(dsv, t, dh, dl);
#pragma unroll
      for (int nt = 0; nt < NTD; ++nt) {
        const typename M::frag kb_ = lds_perm_frag<E, D>(kt, 32 * nt, 32 * kh, t);
        dq[nt] = M::mma(dh, kb_, dq[nt]);
        if constexpr (!M::exact_operands) dq[nt] = M::mma(dl, kb_, dq[nt]);
      }
    }
    if constexpr (D == 128) __builtin_amdgcn_s_setprio(0);
  }

  // sum the two key-half partials: kh = 1 hands its accumulators over in LDS
  __syncthreads();
  float* xch = reinterpret_cast<float*>(&kbuf[0][0]);
  if (kh == 1) {
#pragma unroll
    for (int nt = 0; nt < NTD; ++nt)
#pragma unroll
      for (int r = 0; r < 16; ++r) xch[((qh * NTD + nt) * 16 + r) * 64 + lane] = dq[nt][r];
  }
  __syncthreads();
  if (kh == 1 || !wave_ok) return;
  float* dQ = a.dq + head;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int ir = q0 + crow(r);
    if (ir < n) {
#pragma unroll
      for (int nt = 0; nt < NTD; ++nt)
        dQ[(size_t)ir * D + 32 * nt + (lane & 31)] =
            a.scale * (dq[nt][r] + xch[((qh * NTD + nt) * 16 + r) * 64 + lane]);
    }
  }
}

template <typename E, int D>
hipError_t launch_dkdv_d(const BwdArgs& a, hipStream_t s) {
  // d = 128 bf16 takes the column-split kernel; at d = 64 (and for fp32)
  // the one-block kernel already runs two waves per SIMD without the union
  // of two query-block lists, and is faster on sparse masks.
  if constexpr (sizeof(E) == 2 && D == 128) {
    dim3 grid((unsigned)(a.BH * ((a.T + 1) / 2))), block(BWD2_NT);
    auto kernel = dkdv2_kernel<D, 0>;
    if (a.gk == 1) kernel = dkdv2_kernel<D, 1>;
    if (a.gk == 2) kernel = dkdv2_kernel<D, 2>;
    if (a.gk == 4) kernel = dkdv2_kernel<D, 4>;
    return launch_kernel(kernel, grid, block, s, a);
  }
  dim3 grid((unsigned)(a.BH * a.T)), block(BWD_NT);
  auto kernel = dkdv_kernel<E, D, 0>;
  if (a.gk == 1) kernel = dkdv_kernel<E, D, 1>;
  if (a.gk == 2) kernel = dkdv_kernel<E, D, 2>;
  if (a.gk == 4) kernel = dkdv_kernel<E, D, 4>;
  return launch_kernel(kernel, grid, block, s, a);
}

template <typename E, int D>
hipError_t launch_dq_d(const BwdArgs& a, hipStream_t s) {
  dim3 grid((unsigned)(a.BH * a.T)), block(DQ_NT);
  auto kernel = dq_kernel<E, D, 0>;
  if (a.gk == 1) kernel = dq_kernel<E, D, 1>;
  if (a.gk == 2) kernel = dq_kernel<E, D, 2>;
  if (a.gk == 4) kernel = dq_kernel<E, D, 4>;
  return launch_kernel(kernel, grid, block, s, a);
}

template <typename E, int D>
hipError_t launch_delta_d(const DeltaArgs& a, hipStream_t s) {
  dim3 grid((unsigned)((a.rows + 15) / 16)), block(256);
  return launch_kernel(delta_kernel<E, D>, grid, block, s, a);
}

}  // namespace

hipError_t launch_delta(const DeltaArgs& a, int dtype, int head_dim, hipStream_t s) {
  if (dtype == 0) return head_dim == 64 ? launch_delta_d<__bf16, 64>(a, s) : launch_delta_d<__bf16, 128>(a, s);
  return head_dim == 64 ? launch_delta_d<float, 64>(a, s) : launch_delta_d<float, 128>(a, s);
}

hipError_t launch_bwd_dkdv(const BwdArgs& a, int dtype, int head_dim, hipStream_t s) {
  if (dtype == 0) return head_dim == 64 ? launch_dkdv_d<__bf16, 64>(a, s) : launch_dkdv_d<__bf16, 128>(a, s);
  return head_dim == 64 ? launch_dkdv_d<float, 64>(a, s) : launch_dkdv_d<float, 128>(a, s);
}

hipError_t launch_bwd_dq(const BwdArgs& a, int dtype, int head_dim, hipStream_t s) {
  if (dtype == 0) return head_dim == 64 ? launch_dq_d<__bf16, 64>(a, s) : launch_dq_d<__bf16, 128>(a, s);
  return head_dim == 64 ? launch_dq_d<float, 64>(a, s) : launch_dq_d<float, 128>(a, s);
}

}  // namespace ea
