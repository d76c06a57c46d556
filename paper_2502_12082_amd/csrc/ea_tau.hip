// ea_tau.hip -- per-row alpha-entmax threshold tau and the 64x64 block mask.
//
// Method (Sec. 3.1 Algorithm 1, block form Algorithm 3 of App. A): for each
// query row i, x_ij = (alpha-1) * scale * <q_i, k_j>; tau_i is the root of
// f(tau) = sum_j [x_ij - tau]_+^gamma - 1 (Eq. 3).  f, f', f'' (Eq. 3, 6, 7)
// are additive over key blocks, so each pass streams K once and accumulates
// three per-row sums; between passes the bracket is updated with the
// bisection rule B_f (Eq. 4) and the Halley step H_f (Eq. 5) is taken when it
// lands inside the bracket, otherwise the midpoint.  The bracket starts at
// [max_j x_ij - 1, max_j x_ij - n_i^(1-alpha)] after a first pass that finds
// the row maximum.  The block mask of Eq. 8 is recorded during every
// evaluation pass; the pass at the returned tau is the last one, so the mask
// describes exactly the probabilities that the forward and backward kernels
// recompute from that tau.
//
// Layout on gfx950: one workgroup = 4 waves = 128 query rows (two mask
// rows); each wave keeps its 32 query rows as MFMA B operands in registers
// and computes S^T tiles (keys x queries), so every lane owns one query and
// the per-row sums stay in-lane until the end of a pass.  K tiles of 64 keys
// are copied into a double-buffered LDS tile by global_load_lds, the next
// one in flight while the current one is consumed.  A workgroup stops as
// soon as every row it owns has |f(tau)| <= tol, or after max_iter updates.
#include <type_traits>

#include "ea_common.h"
#include "ea_internal.h"

namespace ea {

namespace {

constexpr int TAU_WAVES = 4;
constexpr int TAU_NT = 64 * TAU_WAVES;
constexpr int TAU_ROWS = 32 * TAU_WAVES;

// MODE: SOLVE writes tau, the block mask and stats; FUSED_O (inference) and
// FUSED_O2 (training) are the no-mask forward of Algorithm 2: once tau is
// known, the same workgroup streams K and V once more and writes O (and
// O2), with no mask or tables.
constexpr int SOLVE = 0, FUSED_O = 1, FUSED_O2 = 2;

template <typename E, int D, int GK, int MODE>
__global__ __launch_bounds__(TAU_NT, MODE == SOLVE ? 4 : 2) void tau_solve_kernel(TauArgs a) {
  using TL = PadTile<E, D>;
  using TV = Tile<E, D>;
  using M = Mma<E>;
  constexpr int KS = D / M::KW;
  constexpr int NTD = D / 32;
  constexpr int PS = perm_steps<E>();
  constexpr bool FUSED = MODE != SOLVE, TRAIN = MODE == FUSED_O2;
  constexpr int BW = MAX_KEY_BLOCKS / 32;  // mask words per wave
  __shared__ __attribute__((aligned(16))) E kbuf[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) E vbuf[FUSED ? 2 : 1][FUSED ? TV::ELEMS : 8];
  // bit kb of word kb / 32: key block kb holds a positive probability for
  // one of the wave's 32 rows
  __shared__ uint32_t bits[TAU_WAVES * BW];

  const int lane = lane_id(), w = wave_id();
  const int n = a.n, T = a.T;
  const int nqt = (n + TAU_ROWS - 1) / TAU_ROWS;
  const int TW = (T + 31) / 32;
  const float c = a.c, g = a.gamma;
  // The Newton step from any tau is a lower bound of the root when f is
  // convex, i.e. gamma >= 1 (alpha <= 2).
  const bool newton_bound = g >= 1.f;
  // This workgroup's slot of the candidate cache (entry e of thread t at
  // [e * TAU_NT + t]), or null when the workspace has no slot for it.
  const int tile = blockIdx.x;
  CandEntry* const cache =
      a.cand && tile < a.slots ? a.cand + (size_t)tile * a.cap * TAU_NT : nullptr;

  TileDma<TL, D, TAU_NT> dma;
  dma.init();

  {
    const int bh = tile % a.BH;
    int qt = tile / a.BH;
    if (a.causal) qt = nqt - 1 - qt;  // longest rows first
    const int q0 = qt * TAU_ROWS + 32 * w;
    const int i = q0 + (lane & 31);
    const bool row_ok = i < n;
    const int ni = a.causal ? i + 1 : n;
    const E* Q = static_cast<const E*>(a.q) + (size_t)bh * n * D;
    const E* K = static_cast<const E*>(a.k) + (size_t)bh * n * D;

    const int wg_last = min(n, (qt + 1) * TAU_ROWS) - 1;
    const int nkb = a.causal ? wg_last / BLK + 1 : T;
    const int wave_last = min(n - 1, q0 + 31);
    const bool wave_ok = q0 < n;

    typename M::frag qf[KS];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[kk] = load_row_frag_global<E, D>(Q, i, n, kk);

    for (int x = threadIdx.x; x < TAU_WAVES * TW; x += TAU_NT) bits[(x / TW) * BW + (x % TW)] = 0;

    // Streams every key block the tile needs, double-buffered: block kb + 1
    // is copied into LDS while `body(kb, tile)` works on block kb.
    auto stream = [&](auto&& body) {
      dma.issue(kbuf[0], K, 0, n);
      for (int kb = 0; kb < nkb; ++kb) {
        dma_wait();
        __syncthreads();
        if (kb + 1 < nkb) dma.issue(kbuf[(kb + 1) & 1], K, (kb + 1) * BLK, n);
        body(kb, kbuf[kb & 1]);
      }
      __syncthreads();  // the next pass refills buffer 0
    };

    // S^T sub-tiles of the staged block: keys [0, 32) and [32, 64) x this
    // wave's 32 queries; value r of lane l is key 32 sub + crow(r), query
    // l%32.  The two accumulation chains are interleaved so neither waits on
    // the other.
    auto scores = [&](const E* kt, f32x16& s0, f32x16& s1) {
      s0 = zero16();
      s1 = zero16();
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const typename M::frag a0 = lds_row_frag_pad<E, D>(kt, (lane & 31), kk);
        const typename M::frag a1 = lds_row_frag_pad<E, D>(kt, 32 + (lane & 31), kk);
        s0 = M::mma(a0, qf[kk], s0);
        s1 = M::mma(a1, qf[kk], s1);
      }
    };
    // Sub-tile state for the calling wave: 0 = nothing valid, 1 = all valid,
    // 2 = needs per-element masking (ragged tail or causal diagonal).
    auto sub_kind = [&](int j0) {
      if (!wave_ok || j0 >= n || (a.causal && j0 > wave_last)) return 0;
      if (j0 + 31 >= n || (a.causal && j0 + 31 > q0)) return 2;
      return 1;
    };
    auto valid = [&](int j) { return j < n && (!a.causal || j <= i); };
    // Invalid keys of a masked sub-tile become -inf: they cannot be the
    // maximum, and the clamp of [x - tau]_+ turns them into exactly 0.
    auto mask_tile = [&](f32x16& s, int j0) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (!valid(j0 + crow(r))) s[r] = -INFINITY;
    };

    // ---- pass 0: row maximum of the raw scores (scale > 0, so the maximum
    // of x = c s is c times the maximum of s)
    float smax = -INFINITY;
    auto max_tile = [&](const f32x16& s) {
#pragma unroll
      for (int r = 0; r < 16; r += 2) smax = fmaxf(smax, fmaxf(s[r], s[r + 1]));
    };
    stream([&](int kb, const E* kt) {
      const int j0 = kb * BLK;
      const int k0 = sub_kind(j0), k1 = sub_kind(j0 + 32);
      if (k0 == 0 && k1 == 0) return;
      f32x16 s0, s1;
      scores(kt, s0, s1);
      if (k0 == 1 && k1 == 1) {
        max_tile(s0);
        max_tile(s1);
        return;
      }
      if (k0 == 2) mask_tile(s0, j0);
      if (k1 == 2) mask_tile(s1, j0 + 32);
      if (k0) max_tile(s0);
      if (k1) max_tile(s1);
    });
    smax = fmaxf(smax, __shfl_xor(smax, 32));

    float lo = 0.f, hi = 0.f, tau = 0.f;
    if (row_ok) {
      const float m = c * smax;
      lo = m - 1.f;
      hi = m - powf((float)ni, 1.f - a.alpha);
      tau = 0.5f * (lo + hi);
    }

    int passes = 1;      // K passes (streamed), the max pass included
    bool cached = false; // evaluations run on the candidate cache
    int attempts = 0;    // cache fills tried
    int cc = 0;          // candidates this thread found in the last fill
    int cmax = 0;        // wave maximum of cc once the cache is in use
    bool small_support = false;  // every thread's support count <= cap / 2
    float f_prev = INFINITY;     // |f| at the previous evaluation
    float usum = 0.f;            // sum of u = z^(gamma-1) over the row at the last tau
    for (int it = 0;; ++it) {
      // ---- evaluation at tau: m0 = sum z^gamma, m1 = sum z^(gamma-1),
      // m2 = sum z^(gamma-2) over the strict support z > 0, and mc = the size
      // of the support (for gamma = 1, 2 that is the last sum, counted exactly
      // as an integer).
      float m0 = 0.f, m1 = 0.f, m2 = 0.f;
      int mc = 0;
      // Adds the terms of one value z = [x - tau]_+ (clamped to [0, 1]) to
      // (t0, t1, t2, tc).
      auto add_z = [&](float zp, float& t0, float& t1, float& t2, int& tc) {
        if constexpr (GK == 1) {
          t0 += zp;
          tc += in_support(zp);
        } else if constexpr (GK == 2) {
          t0 = fmaf(zp, zp, t0);
          t1 += zp;
          tc += in_support(zp);
        } else if constexpr (GK == 4) {
          const float z2 = zp * zp;
          t0 = fmaf(z2, z2, t0);
          t1 = fmaf(z2, zp, t1);
          t2 += z2;
          tc += in_support(zp);
        } else {
          if (zp > 0.f) {
            const float l = __log2f(zp);
            t0 += exp2f(g * l);
            t1 += exp2f((g - 1.f) * l);
            t2 += exp2f((g - 2.f) * l);
            ++tc;
          }
        }
      };
      // Adds one sub-tile; returns whether it holds a positive probability.
      auto eval_tile = [&](const f32x16& s) {
        if constexpr (GK == 1 || GK == 2) {
          int cnt = 0;
#pragma unroll
          for (int r = 0; r < 16; r += 2) {
            const float za = relu_z(c, s[r], tau), zb = relu_z(c, s[r + 1], tau);
            if constexpr (GK == 1) {
              m0 += za;
              m0 += zb;
            } else {
              m0 = fmaf(za, za, m0);
              m0 = fmaf(zb, zb, m0);
              m1 += za;
              m1 += zb;
            }
            cnt += in_support(za) + in_support(zb);
          }
          mc += cnt;
          return cnt > 0;
        } else {
          // tile sums start from 0, so t0 > 0 exactly when some term is > 0
          float t0 = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r) add_z(relu_z(c, s[r], tau), t0, m1, m2, mc);
          m0 += t0;
          return t0 > 0.f;
        }
      };
      // Appends the entries x > lo of a sub-tile to this thread's cache list.
      // Every later tau stays >= lo, so the entries left out are 0 there.
      const float s_lo = row_ok ? lo / c : INFINITY;  // rows past n collect nothing
      CandEntry* const mine = cache + threadIdx.x;
      auto fill_tile = [&](const f32x16& s, int kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if (s[r] > s_lo) {
            if (cc < a.cap) mine[cc * TAU_NT] = CandEntry{c * s[r], kb};
            ++cc;
          }
        }
      };

      // From the second evaluation on, a tile with a cache slot tries (at
      // most twice) to collect its candidates x > lo in a K pass of their
      // own, when the last streamed evaluation suggests that they fit; the
      // evaluation at tau then runs on the cache.  If a thread's list
      // overflows, this evaluation streams K as usual.
      if (!cached && cache && it >= 1 && attempts < 2 && small_support) {
        ++attempts;
        cc = 0;
        stream([&](int kb, const E* kt) {
          const int j0 = kb * BLK;
          const int k0 = sub_kind(j0), k1 = sub_kind(j0 + 32);
          if (k0 == 0 && k1 == 0) return;
          f32x16 s0, s1;
          scores(kt, s0, s1);
          if (k0 == 2) mask_tile(s0, j0);
          if (k1 == 2) mask_tile(s1, j0 + 32);
          if (k0) fill_tile(s0, kb);
          if (k1) fill_tile(s1, kb);
        });
        ++passes;
        if (!__syncthreads_or(cc > a.cap)) {
          cached = true;
          cmax = cc;
#pragma unroll
          for (int o = 32; o >= 1; o >>= 1) cmax = max(cmax, __shfl_xor(cmax, o));
        }
      }
      if (!cached) {
        // streamed evaluation; the mask bits of every block are rewritten
        uint32_t word = 0;  // mask bits of the current 32-block group (wave-uniform)
        stream([&](int kb, const E* kt) {
          const int j0 = kb * BLK;
          const int k0 = sub_kind(j0), k1 = sub_kind(j0 + 32);
          bool any = false;
          if (k0 == 1 && k1 == 1) {  // every key valid: one straight-line block
            f32x16 s0, s1;
            scores(kt, s0, s1);
            const bool a0 = eval_tile(s0);
            const bool a1 = eval_tile(s1);
            any = a0 || a1;
          } else if (k0 != 0 || k1 != 0) {
            f32x16 s0, s1;
            scores(kt, s0, s1);
            if (k0 == 2) mask_tile(s0, j0);
            if (k1 == 2) mask_tile(s1, j0 + 32);
            if (k0) any |= eval_tile(s0);
            if (k1) any |= eval_tile(s1);
          }
          if (__ballot(any) != 0ull) word |= 1u << (kb & 31);
          if ((kb & 31) == 31 || kb == nkb - 1) {
            if (lane == 0) bits[w * BW + (kb >> 5)] = word;
            word = 0;
          }
        });
        ++passes;
        // support sizes at this tau, a guide to the size of the candidate lists
        small_support = !__syncthreads_or(mc > a.cap / 2);
      } else {
        // cached evaluation: the same sums over this thread's list
        for (int e = 0; e < cmax; ++e) {
          if (e < cc) {
            const CandEntry ce = cache[(size_t)e * TAU_NT + threadIdx.x];
            add_z(__builtin_amdgcn_fmed3f(ce.x - tau, 0.f, 1.f), m0, m1, m2, mc);
          }
        }
      }
      if constexpr (GK == 1) m1 = (float)mc;
      if constexpr (GK == 2) m2 = (float)mc;
      m0 += __shfl_xor(m0, 32);
      m1 += __shfl_xor(m1, 32);
      m2 += __shfl_xor(m2, 32);
      usum = m1;

      const float f = m0 - 1.f;                        // Eq. 3
      float f1, f2;                                    // Eq. 6, 7
      if constexpr (GK == 1) {
        f1 = -m1;
        f2 = 0.f;
      } else if constexpr (GK == 2) {
        f1 = -2.f * m1;
        f2 = 2.f * m2;
      } else if constexpr (GK == 4) {
        f1 = -4.f * m1;
        f2 = 12.f * m2;
      } else {
        f1 = -g * m1;
        f2 = g * (g - 1.f) * m2;
      }
      const bool conv = !row_ok || fabsf(f) <= a.tol;
      if (__syncthreads_and(conv) || it >= a.max_iter) break;
      if (row_ok) {
        if (f < 0.f)  // B_f, Eq. 4 ("otherwise" branch when f == 0)
          hi = tau;
        else
          lo = tau;
        // Bracket test of Algorithm 1 with fp32 rounding: when the root sits
        // on an end of the bracket (one-hot rows: tau = max - 1; constant
        // rows: tau = max - n^(1-alpha)) the Halley value lands within a few
        // ulps on either side of it, so values within `slack` are accepted
        // and clamped into [lo, hi].  NaN and inf fail the test and take the
        // midpoint.
        const float slack = 1e-6f * fmaxf(1.f, fmaxf(fabsf(lo), fabsf(hi)));
        if (newton_bound && f1 < 0.f) {
          // convexity: the tangent at tau meets zero at or below the root;
          // a margin of 10 slacks covers the rounding of that point
          const float tn = tau - f / f1 - 10.f * slack;
          lo = fminf(fmaxf(lo, tn), hi);
        }
        const float th = tau - 2.f * f * f1 / (2.f * f1 * f1 - f * f2);  // H_f, Eq. 5
        bool take = th >= lo - slack && th <= hi + slack;
        // For gamma < 1 (alpha > 2) f' diverges at every kink x_j, and H_f can
        // creep towards a kink in ever smaller steps that all stay inside
        // the bracket, so the fail-safe above never fires.  There the
        // midpoint is also taken whenever |f| has not halved since the last
        // evaluation, which bounds the bracket's shrinkage from below.
        if (!newton_bound && fabsf(f) > 0.5f * f_prev) take = false;
        f_prev = fabsf(f);
        tau = take ? fminf(fmaxf(th, lo), hi) : 0.5f * (lo + hi);
      }
    }

    if (row_ok && lane < 32) a.tau[(size_t)bh * n + i] = tau;

    if constexpr (FUSED) {
      // ---- Algorithm 2 at the returned tau: O = sum_j P_ij V_j, and in
      // training O2 = sum_j u_ij V_j / sum_j u_ij (sum u is the solver's last
      // S1 sum), over every valid key block.
      f32x16 o[NTD], o2[NTD];
#pragma unroll
      for (int t = 0; t < NTD; ++t) {
        o[t] = zero16();
        if constexpr (TRAIN) o2[t] = zero16();
      }
      const E* V = static_cast<const E*>(a.v) + (size_t)bh * n * D;
      TileDma<TV, D, TAU_NT> vdma;
      vdma.init();
      auto pv_tile = [&](const f32x16& s, const E* vt, int sub) {
        float p[16], u[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float zp = relu_z(c, s[r], tau);
          if constexpr (TRAIN)
            Gamma<GK>::pu(zp, g, p[r], u[r]);
          else
            p[r] = Gamma<GK>::p_only(zp, g);
        }
#pragma unroll
        for (int t = 0; t < PS; ++t) {
          const typename M::frag pa = M::pack(p, t);
          typename M::frag uh, ul;
          if constexpr (TRAIN) M::pack_split(u, t, uh, ul);
#pragma unroll
          for (int nt = 0; nt < NTD; ++nt) {
            const typename M::frag vb = lds_perm_frag<E, D>(vt, 32 * nt, 32 * sub, t);
            o[nt] = M::mma(pa, vb, o[nt]);
            if constexpr (TRAIN) {
              o2[nt] = M::mma(uh, vb, o2[nt]);
              if constexpr (!M::exact_operands) o2[nt] = M::mma(ul, vb, o2[nt]);
            }
          }
        }
      };
      dma.issue(kbuf[0], K, 0, n);
      vdma.issue(vbuf[0], V, 0, n);
      for (int kb = 0; kb < nkb; ++kb) {
        dma_wait();
        __syncthreads();
        if (kb + 1 < nkb) {
          dma.issue(kbuf[(kb + 1) & 1], K, (kb + 1) * BLK, n);
          vdma.issue(vbuf[(kb + 1) & 1], V, (kb + 1) * BLK, n);
        }
        const int j0 = kb * BLK;
        const int k0 = sub_kind(j0), k1 = sub_kind(j0 + 32);
        if (k0 == 0 && k1 == 0) continue;
        f32x16 s0, s1;
        scores(kbuf[kb & 1], s0, s1);
        if (k0 == 2) mask_tile(s0, j0);
        if (k1 == 2) mask_tile(s1, j0 + 32);
        if (k0) pv_tile(s0, vbuf[kb & 1], 0);
        if (k1) pv_tile(s1, vbuf[kb & 1], 1);
      }
      if (!wave_ok) return;
      // accumulator value r of lane l: query q0 + crow(r), column 32 nt + l % 32
      E* O = static_cast<E*>(a.o) + (size_t)bh * n * D;
      float* O2 = TRAIN ? a.o2 + (size_t)bh * n * D : nullptr;
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
      return;
    }

    if (cached) {
      // mask bits at the returned tau from the cached entries
      for (int x = lane; x < TW; x += 64) bits[w * BW + x] = 0;
      __syncthreads();
      for (int e = 0; e < cmax; ++e) {
        if (e < cc) {
          const CandEntry ce = cache[(size_t)e * TAU_NT + threadIdx.x];
          if (ce.x - tau > 0.f) atomicOr(&bits[w * BW + (ce.kb >> 5)], 1u << (ce.kb & 31));
        }
      }
    }

    __syncthreads();
    constexpr int QBLOCKS = TAU_WAVES / 2;  // 64-row mask rows per workgroup
    for (int x = threadIdx.x; x < QBLOCKS * T; x += TAU_NT) {
      const int half = x / T, kb = x % T;
      const int qb = QBLOCKS * qt + half;
      if (qb < T) {
        const uint32_t both = bits[(2 * half) * BW + (kb >> 5)] | bits[(2 * half + 1) * BW + (kb >> 5)];
        const uint8_t b = (both >> (kb & 31)) & 1u;
        a.mask[((size_t)bh * T + qb) * T + kb] = b;
        if (a.stats && kb == 0) a.stats[(size_t)bh * T + qb] = passes;
      }
    }
  }
}

template <typename E, int D, int MODE>
hipError_t launch_tau_d(const TauArgs& a, hipStream_t s) {
  dim3 grid((unsigned)(a.BH * ((a.n + TAU_ROWS - 1) / TAU_ROWS))), block(TAU_NT);
  auto kernel = tau_solve_kernel<E, D, 0, MODE>;
  if (a.gk == 1) kernel = tau_solve_kernel<E, D, 1, MODE>;
  if (a.gk == 2) kernel = tau_solve_kernel<E, D, 2, MODE>;
  if (a.gk == 4) kernel = tau_solve_kernel<E, D, 4, MODE>;
  return launch_kernel(kernel, grid, block, s, a);
}

template <int MODE>
hipError_t launch_tau_mode(const TauArgs& a, int dtype, int head_dim, hipStream_t s) {
  if (dtype == 0)
    return head_dim == 64 ? launch_tau_d<__bf16, 64, MODE>(a, s) : launch_tau_d<__bf16, 128, MODE>(a, s);
  return head_dim == 64 ? launch_tau_d<float, 64, MODE>(a, s) : launch_tau_d<float, 128, MODE>(a, s);
}

}  // namespace

hipError_t launch_tau(const TauArgs& a, int dtype, int head_dim, hipStream_t s) {
  return launch_tau_mode<SOLVE>(a, dtype, head_dim, s);
}

hipError_t launch_tau_fused(const TauArgs& a, int dtype, int head_dim, hipStream_t s) {
  return a.o2 ? launch_tau_mode<FUSED_O2>(a, dtype, head_dim, s)
              : launch_tau_mode<FUSED_O>(a, dtype, head_dim, s);
}

}  // namespace ea
