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
// the row maximum; that pass also raises the lower end with the largest
// scores' own bound (see pass 0) and, given a workspace, collects each row's
// scores above it, on which every later evaluation can run without K.  The
// masked path's block mask of Eq. 8 is recorded during every streamed
// evaluation (or rebuilt from the collected scores) at the returned tau, so
// the mask describes exactly the probabilities that the forward and backward
// kernels recompute from that tau.
//
// Two kernels.  solve_kernel is the masked path's solver (tau, the block
// mask and stats; its layout is described where it is defined).
// tau_solve_kernel is the no-mask forward: the same solver followed, in the
// same workgroup, by the O (and O2) pass of Algorithm 2.  Its layout on
// gfx950: one workgroup = 4 waves = 128 query rows; each wave keeps its 32
// query rows as MFMA B operands in registers and computes S^T tiles (keys x
// queries), so every lane owns one query and the per-row sums stay in-lane
// until the end of a pass.  In both, K tiles of 64 keys are copied into a
// double-buffered LDS tile by global_load_lds, the next one in flight while
// the current one is consumed, and a workgroup stops as soon as every row it
// owns has |f(tau)| <= tol, or after max_iter updates.
#include <type_traits>

#include "ea_common.h"
#include "ea_internal.h"

namespace ea {

namespace {

constexpr int TAU_WAVES = 4;
constexpr int TAU_NT = 64 * TAU_WAVES;
constexpr int TAU_ROWS = 32 * TAU_WAVES;

// MODE: FUSED_O (inference) and FUSED_O2 (training) are the no-mask forward
// of Algorithm 2: once tau is known, the same workgroup streams K and V once
// more and writes O (and O2), with no mask or tables.
constexpr int FUSED_O = 1, FUSED_O2 = 2;

template <typename E, int D, int GK, int MODE>
__global__ __launch_bounds__(TAU_NT, 2) void tau_solve_kernel(TauArgs a) {
  using TL = PadTile<E, D>;
  using TV = Tile<E, D>;
  using M = Mma<E>;
  constexpr int KS = D / M::KW;
  constexpr int NTD = D / 32;
  constexpr int PS = perm_steps<E>();
  constexpr bool TRAIN = MODE == FUSED_O2;
  __shared__ __attribute__((aligned(16))) E kbuf[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) E vbuf[2][TV::ELEMS];

  const int lane = lane_id(), w = wave_id();
  const int n = a.n, T = a.T;
  const int nqt = (n + TAU_ROWS - 1) / TAU_ROWS;
  const float c = a.c, g = a.gamma;
  // The Newton step from any tau is a lower bound of the root when f is
  // convex, i.e. gamma >= 1 (alpha <= 2).
  const bool newton_bound = g >= 1.f;
  // Tile a.tile0 + blockIdx.x, and this workgroup's slot of the candidate
  // cache (entry e of thread t at [e * TAU_NT + t]), or null when the
  // workspace has no slot for it.  A launch covers at most one tile per slot
  // (see launch_tiles).
  const int tile = a.tile0 + (int)blockIdx.x;
  CandEntry* const cache = a.cand && (int)blockIdx.x < a.slots
                               ? static_cast<CandEntry*>(a.cand) + (size_t)blockIdx.x * a.cap * TAU_NT
                               : nullptr;

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
    // of x = c s is c times the maximum of s), and a tighter lower end of
    // the bracket: if j distinct keys score at least v, each of their terms
    // of f is at least (c v - tau)^gamma at any tau below c v, so at the root
    // j (c v - tau)^gamma <= 1 and tau >= c v - j^(-1/gamma).  j = 1 with v
    // the maximum is Algorithm 1's tau >= max - 1.  Each lane keeps the four
    // largest maxima of its 16-score sub-tile columns (each over keys of its
    // own); the two lanes of a row merge theirs into the row's eight largest,
    // and v_j is the j-th of those.
    float t4[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};  // descending
    auto tile_max = [&](const f32x16& s) {
      float v = fmaxf(s[0], s[1]);
#pragma unroll
      for (int r = 2; r < 16; r += 2) v = fmaxf(v, fmaxf(s[r], s[r + 1]));
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float h = fmaxf(t4[j], v);
        v = fminf(t4[j], v);
        t4[j] = h;
      }
    };
    stream([&](int kb, const E* kt) {
      const int j0 = kb * BLK;
      const int k0 = sub_kind(j0), k1 = sub_kind(j0 + 32);
      if (k0 == 0 && k1 == 0) return;
      f32x16 s0, s1;
      scores(kt, s0, s1);
      if (k0 == 2) mask_tile(s0, j0);
      if (k1 == 2) mask_tile(s1, j0 + 32);
      if (k0) tile_max(s0);
      if (k1) tile_max(s1);
    });

    float lo = 0.f, hi = 0.f, tau = 0.f;
    {
      // the row's eight largest sub-tile maxima, descending: the two lanes'
      // sorted lists merged by Batcher's odd-even network
      float u[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        u[j] = t4[j];
        u[4 + j] = __shfl_xor(t4[j], 32);
      }
      auto cx = [&](int x, int y) {
        const float h = fmaxf(u[x], u[y]);
        u[y] = fminf(u[x], u[y]);
        u[x] = h;
      };
      cx(0, 4); cx(1, 5); cx(2, 6); cx(3, 7);
      cx(2, 4); cx(3, 5);
      cx(1, 2); cx(3, 4); cx(5, 6);
      if (row_ok) {
        const float m = c * u[0];
        hi = m - powf((float)ni, 1.f - a.alpha);
        float b = m - 1.f;
#pragma unroll
        for (int j = 1; j < 8; ++j) b = fmaxf(b, fmaf(c, u[j], -exp2f(-__log2f((float)(j + 1)) / g)));
        // For gamma >= 1, two Newton steps on f restricted to these eight
        // scores: that f is convex and decreasing, so the steps stay below
        // its root, which is below tau (the dropped terms are >= 0).  Every z
        // is at most 1 and z_1 > 0, so the derivative is nonzero.
        if (g >= 1.f) {
#pragma unroll
          for (int it = 0; it < 2; ++it) {
            float f = -1.f, fp = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const float z = fmaf(c, u[j], -b);
              if (z > 0.f) {
                float pj, uj;
                Gamma<GK>::pu(z, g, pj, uj);
                f += pj;
                fp += uj;
              }
            }
            b += f / (g * fp);
          }
        }
        // the bound may round above the root by a few ulps (rows whose whole
        // support is among the eight reach it)
        lo = fminf(b - 4e-6f * fmaxf(1.f, fabsf(b)), hi);
        tau = 0.5f * (lo + hi);
      }
    }

    bool cached = false; // evaluations run on the candidate cache
    int attempts = 0;    // cache fills tried
    int cc = 0;          // candidates this thread found in the last fill
    int cmax = 0;        // wave maximum of cc once the cache is in use
    __shared__ int fill_full;  // some list of the current fill overflowed
    CandEntry* const mine = cache ? cache + threadIdx.x : nullptr;
    // Reads this thread's list in batches of eight independent loads and
    // calls `use` on each entry; the trip count is the wave's longest list.
    auto scan = [&](auto&& use) {
      for (int e0 = 0; e0 < cmax; e0 += 8) {
        CandEntry ce[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (e0 + u < cc) ce[u] = mine[(size_t)(e0 + u) * TAU_NT];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (e0 + u < cc) use(ce[u]);
      }
    };
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
      // Adds one sub-tile to the sums.
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
        } else {
          float t0 = 0.f;  // summed per tile, then added to the row sum
#pragma unroll
          for (int r = 0; r < 16; ++r) add_z(relu_z(c, s[r], tau), t0, m1, m2, mc);
          m0 += t0;
        }
      };
      // Appends the entries x > lo of a sub-tile to this thread's cache list.
      // Every later tau stays >= lo, so the entries left out are 0 there.
      // The threshold in score units carries a margin for the rounding of
      // lo / c (a superset of the entries is harmless).
      const float s_lo0 = lo / c;
      const float s_lo = row_ok ? s_lo0 - 1e-6f * fmaxf(fabsf(s_lo0), 1.f / c) : INFINITY;
      auto fill_tile = [&](const f32x16& s, int jb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if (s[r] > s_lo) {
            if (cc < a.cap) mine[(size_t)cc * TAU_NT] = CandEntry{s[r], jb + crow(r)};
            ++cc;
          }
        }
      };
      // Decides, after a fill, whether every list fit.
      auto fill_done = [&]() {
        if (!__syncthreads_or(cc > a.cap)) {
          cached = true;
          cmax = cc;
#pragma unroll
          for (int o = 32; o >= 1; o >>= 1) cmax = max(cmax, __shfl_xor(cmax, o));
        }
      };

      // A tile with a cache slot collects its candidates x > lo during the
      // first evaluation; if a list overflows, it tries (once more) later in
      // a K pass of its own, when the last streamed evaluation suggests that
      // they fit, and that evaluation then runs on the cache.  Otherwise the
      // evaluation streams K.
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
          if (k0) fill_tile(s0, j0);
          if (k1) fill_tile(s1, j0 + 32);
        });
        fill_done();
      }
      if (!cached) {
        // streamed evaluation
        const bool fill = cache && it == 0;
        if (fill) {
          ++attempts;
          cc = 0;
          if (threadIdx.x == 0) fill_full = 0;  // read after the first block's barrier
        }
        stream([&](int kb, const E* kt) {
          const int j0 = kb * BLK;
          const int k0 = sub_kind(j0), k1 = sub_kind(j0 + 32);
          // once a list of this fill has overflowed, no thread stores more
          const bool fill_now = fill && !fill_full;
          if (k0 == 1 && k1 == 1) {  // every key valid: one straight-line block
            f32x16 s0, s1;
            scores(kt, s0, s1);
            eval_tile(s0);
            eval_tile(s1);
            if (fill_now) {
              fill_tile(s0, j0);
              fill_tile(s1, j0 + 32);
            }
          } else if (k0 != 0 || k1 != 0) {
            f32x16 s0, s1;
            scores(kt, s0, s1);
            if (k0 == 2) mask_tile(s0, j0);
            if (k1 == 2) mask_tile(s1, j0 + 32);
            if (k0) eval_tile(s0);
            if (k1) eval_tile(s1);
            if (fill_now) {
              if (k0) fill_tile(s0, j0);
              if (k1) fill_tile(s1, j0 + 32);
            }
          }
          if (fill_now && cc > a.cap) fill_full = 1;
        });
        // support sizes at this tau, a guide to the size of the candidate lists
        small_support = !__syncthreads_or(mc > a.cap / 2);
        if (fill) {
          if (fill_full) cc = a.cap + 1;  // the fill stopped early: its lists are incomplete
          fill_done();
        }
      } else {
        // cached evaluation: the same sums over this thread's list
        scan([&](const CandEntry& ce) {
          add_z(relu_z(c, ce.s, tau), m0, m1, m2, mc);
        });
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

    // fp32 inputs, general alpha (ea_common.h): tau refined in fp64 by Newton
    // steps on f (Eq. 3, 6) over every entry above the lower edge of the band
    // around the support edge, each with its fp64 score, as in solve_kernel.
    constexpr bool PRECISE = precise_path<E, GK>();
    double tau64 = tau;
    [[maybe_unused]] const float band = PRECISE_BAND * fmaxf(1.f, fabsf(tau));
    [[maybe_unused]] const float* Qf = reinterpret_cast<const float*>(Q);
    [[maybe_unused]] const float* Kf = reinterpret_cast<const float*>(K);
    if constexpr (PRECISE) {
      // use(fp32 score, key) for every valid entry of this lane's row
      auto visit = [&](auto&& use) {
        if (cached) {
          scan([&](const CandEntry& ce) { use(ce.s, ce.j); });
        } else {
          stream([&](int kb, const E* kt) {
            const int j0 = kb * BLK;
            const int k0 = sub_kind(j0), k1 = sub_kind(j0 + 32);
            if (k0 == 0 && k1 == 0) return;
            f32x16 s0, s1;
            scores(kt, s0, s1);
            if (k0 == 2) mask_tile(s0, j0);
            if (k1 == 2) mask_tile(s1, j0 + 32);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              if (k0) use(s0[r], j0 + crow(r));
              if (k1) use(s1[r], j0 + 32 + crow(r));
            }
          });
        }
      };
      for (int it = 0; it < 3; ++it) {
        double t0 = 0.0, t1 = 0.0;
        visit([&](float sv, int jv) {
          if (!row_ok || !(fmaf(c, sv, -tau) > -band)) return;
          const double z = exact_x<D>(Qf + (size_t)i * D, Kf + (size_t)jv * D, a.c64) - tau64;
          if (z > 0.0) {
            t0 += pow(z, a.g64);
            t1 += pow(z, a.g64 - 1.0);
          }
        });
        t0 += __shfl_xor(t0, 32);
        t1 += __shfl_xor(t1, 32);
        if (row_ok && t1 > 0.0) {
          const double slack = 1e-5 * fmax(1.0, fmax(fabs((double)lo), fabs((double)hi)));
          const double tn = tau64 + (t0 - 1.0) / (a.g64 * t1);
          tau64 = fmin(fmax(tn, (double)lo - slack), (double)hi + slack);
        }
      }
    }
    if (row_ok && lane < 32) {
      const float th = (float)tau64;
      a.tau[(size_t)bh * n + i] = th;
      if (a.tau_lo) a.tau_lo[(size_t)bh * n + i] = PRECISE ? (float)(tau64 - (double)th) : 0.f;
    }

    {
      // ---- Algorithm 2 at the returned tau: O = sum_j P_ij V_j, and in
      // training O2 = sum_j u_ij V_j / sum_j u_ij (sum u is the solver's last
      // S1 sum, or, on the fp64 path, the sum of the u this pass forms), over
      // every valid key block.
      f32x16 o[NTD], o2[NTD];
#pragma unroll
      for (int t = 0; t < NTD; ++t) {
        o[t] = zero16();
        if constexpr (TRAIN) o2[t] = zero16();
      }
      const E* V = static_cast<const E*>(a.v) + (size_t)bh * n * D;
      TileDma<TV, D, TAU_NT> vdma;
      vdma.init();
      [[maybe_unused]] float usum_pv = 0.f;  // the fp64 path's sum of u
      auto pv_tile = [&](const f32x16& s, const E* vt, int sub, int j0) {
        float p[16], u[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float zp;
          if constexpr (PRECISE) {
            zp = precise_relu_z<D>(row_ok, c, s[r], tau, band, tau64, Qf + (size_t)i * D,
                                   Kf + (size_t)(j0 + 32 * sub + crow(r)) * D, a.c64);
          } else {
            zp = relu_z(c, s[r], tau);
          }
          if constexpr (TRAIN) {
            Gamma<GK>::pu(zp, g, p[r], u[r]);
            if constexpr (PRECISE) usum_pv += u[r];
          } else {
            p[r] = Gamma<GK>::p_only(zp, g);
          }
        }
#pragma unroll
        for (int t = 0; t < PS; ++t) {
          typename M::frag ph, pl, uh, ul;
          M::pack_split(p, t, ph, pl);
          if constexpr (TRAIN) M::pack_split(u, t, uh, ul);
#pragma unroll
          for (int nt = 0; nt < NTD; ++nt) {
            const typename M::frag vb = lds_perm_frag<E, D>(vt, 32 * nt, 32 * sub, t);
            o[nt] = M::mma(ph, vb, o[nt]);
            if constexpr (!M::exact_operands) o[nt] = M::mma(pl, vb, o[nt]);
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
        if (k0) pv_tile(s0, vbuf[kb & 1], 0, j0);
        if (k1) pv_tile(s1, vbuf[kb & 1], 1, j0);
      }
      if constexpr (PRECISE && TRAIN) usum = usum_pv + __shfl_xor(usum_pv, 32);
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
    }
  }
}

// ----------------------------------------------------------- masked solver
//
// The solver of the masked path (tau, the block mask and stats).  One
// workgroup = 4 waves = 256 query rows; wave w owns the 64-row query block
// qb = 4 qt + w, i.e. one row of the block mask, as two groups of 32 rows
// (g = 0, 1) that are the B operands of its MFMAs.  Every K fragment read
// from LDS feeds two MFMAs (one per group), so a pass reads the K tile from
// LDS half as often per product as with one group per wave; lane l holds
// query l % 32 of each group, so every lane keeps two rows' sums.  The
// evaluation, bracket and cache rules are those of tau_solve_kernel.
constexpr int SV_WAVES = SOLVE_THREADS / 64;
constexpr int SV_NT = SOLVE_THREADS;
constexpr int SV_ROWS = SOLVE_ROWS;
// waves per SIMD for the one-group form (G = 1) of solve_kernel, and the
// grids that use it: fewer 256-row tiles than two per compute unit, and at
// d = 64 rows of up to SV_G1_MAX_N keys
constexpr int SV_OCC1 = 3;
constexpr int SV_G1_BELOW = 512;
constexpr int SV_G1_MAX_N = 32768;
// threads (of SV_NT) with a score above the running bound in one key block
// at or below which the solver's first stream ends early
constexpr int WARM_STOP = SV_NT / 2;
// above it, at d = 64, the first stream covers every key block
constexpr int WARM_ALL = 3 * SV_NT / 4;
static_assert(SV_ROWS == 64 * SV_WAVES, "one 64-row query block per wave (G = 2)");

// G = 2: each wave owns one 64-row query block as two groups of 32 rows.
// G = 1 (small grids): each wave owns 32 rows, two waves share a query
// block, and the workgroup covers 128 rows: twice the waves for the same
// work, with half the state each, so that more of them share each SIMD.
// fp32 operands at d = 128 (128 registers of query fragments) run one wave
// per SIMD with G = 2.
template <typename E, int D, int GK, int G>
__global__ __launch_bounds__(SV_NT, G == 1 ? SV_OCC1 : (sizeof(E) == 4 && D == 128 ? 1 : 2)) void solve_kernel(TauArgs a) {
  using TL = PadTile<E, D>;
  using M = Mma<E>;
  constexpr int KS = D / M::KW;
  constexpr int BW = MAX_KEY_BLOCKS / 32;  // mask words per query block
  constexpr int ROWS = SV_WAVES * 32 * G;  // rows per workgroup
  __shared__ __attribute__((aligned(16))) E kbuf[2][TL::ELEMS];
  // bit kb of word kb / 32: key block kb holds a positive probability for a
  // row of the query block (one per wave with G = 2, per pair of waves with
  // G = 1)
  __shared__ uint32_t bits[SV_WAVES * BW];

  const int lane = lane_id(), w = wave_id();
  const int n = a.n, T = a.T;
  const int nqt = (n + ROWS - 1) / ROWS;
  const int TW = (T + 31) / 32;
  const float c = a.c, g = a.gamma;
  const bool newton_bound = g >= 1.f;  // f convex: Newton steps bound the root from below
  // Tile a.tile0 + blockIdx.x, and this workgroup's cache slot, or none.  A
  // launch covers at most one tile per slot (see launch_tiles).  List
  // (thread t, group gq) holds entry e at index (G e + gq) * SV_NT + t of
  // each array of the slot.  The lists come in three forms:
  //  - quads, as pass 0 collects them: a quad array (16 bytes per entry)
  //    and its key array (2 bytes);
  //  - compacted singles, written by the first cached evaluation from the
  //    quads: a score array (4 bytes) and its key-block array (2 bytes)
  //    after the quad arrays, so that the later evaluations read 4 bytes
  //    per score and the quads stay intact;
  //  - singles of a later fill (CandEntry, 8 bytes), up to `scap` per list
  //    over the whole slot.
  const int tile = a.tile0 + (int)blockIdx.x;
  char* const slot = a.cand && (int)blockIdx.x < a.slots
                         ? static_cast<char*>(a.cand) + (size_t)blockIdx.x * (solve_slot_bytes(a.cap) / 2 * G)
                         : nullptr;
  const bool cache = slot != nullptr;
  char* const kslot = cache ? slot + (size_t)a.cap * G * SV_NT * 16 : nullptr;
  char* const sslot = cache ? kslot + (size_t)a.cap * G * SV_NT * 2 : nullptr;
  char* const bslot = cache ? sslot + (size_t)a.cap * G * SV_NT * 4 : nullptr;
  const int scap = a.cap * (int)(SOLVE_QUAD_BYTES + SOLVE_SINGLE_BYTES) / (int)sizeof(CandEntry);
  const int bh = tile % a.BH;
  int qt = tile / a.BH;
  if (a.causal) qt = nqt - 1 - qt;  // longest rows first
  const int q0 = qt * ROWS + 32 * G * w;  // first row of this wave
  const int qb = q0 / BLK;                 // its query block
  const int qbl = G == 2 ? w : w >> 1;     // that block's mask words in `bits`
  const bool writer = G == 2 || (w & 1) == 0;  // writes the block's mask and stats
  const bool wave_ok = q0 < n;
  int qi[G], ni[G];
  bool row_ok[G];
#pragma unroll
  for (int gq = 0; gq < G; ++gq) {
    qi[gq] = q0 + 32 * gq + (lane & 31);
    row_ok[gq] = qi[gq] < n;
    ni[gq] = a.causal ? qi[gq] + 1 : n;
  }
  const E* Q = static_cast<const E*>(a.q) + (size_t)bh * n * D;
  const E* K = static_cast<const E*>(a.k) + (size_t)bh * n * D;
  const int wg_last = min(n, (qt + 1) * ROWS) - 1;
  const int nkb = a.causal ? wg_last / BLK + 1 : T;

  TileDma<TL, D, SV_NT> dma;
  dma.init();

  typename M::frag qf[G][KS];
#pragma unroll
  for (int gq = 0; gq < G; ++gq)
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[gq][kk] = load_row_frag_global<E, D>(Q, qi[gq], n, kk);

  for (int x = lane; x < TW; x += 64) bits[qbl * BW + x] = 0;

  // Streams every key block in order, double-buffered: block kb + 1 is
  // copied into LDS while body(kb, tile) works on block kb.  The candidate
  // lists keep this order, so a cached evaluation adds the same terms in the
  // same order as a streamed one.
  auto stream_n = [&](int count, auto&& body) {
    dma.issue(kbuf[0], K, 0, n);
    for (int kb = 0; kb < count; ++kb) {
      dma_wait();
      __syncthreads();
      if (kb + 1 < count) dma.issue(kbuf[(kb + 1) & 1], K, (kb + 1) * BLK, n);
      body(kb, kbuf[kb & 1]);
    }
    __syncthreads();  // the next pass refills buffer 0
  };
  auto stream = [&](auto&& body) { stream_n(nkb, body); };
  // Streams every key block once, starting at block `first` and wrapping
  // around.
  auto stream_from = [&](int first, auto&& body) {
    dma.issue(kbuf[0], K, first * BLK, n);
    for (int i = 0; i < nkb; ++i) {
      const int kb = first + i < nkb ? first + i : first + i - nkb;
      const int nx = kb + 1 < nkb ? kb + 1 : 0;
      dma_wait();
      __syncthreads();
      if (i + 1 < nkb) dma.issue(kbuf[(i + 1) & 1], K, nx * BLK, n);
      body(kb, kbuf[i & 1]);
    }
    __syncthreads();  // the next pass refills buffer 0
  };

  // S^T sub-tiles of the staged block: s[h][gq] = keys [32 h, 32 h + 32) x
  // query group gq; value r of lane l is key 32 h + crow(r), query l % 32 of
  // the group.  Four independent accumulation chains.
  auto scores = [&](const E* kt, f32x16 (&s)[2][G]) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int gq = 0; gq < G; ++gq) s[h][gq] = zero16();
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const typename M::frag a0 = lds_row_frag_pad<E, D>(kt, (lane & 31), kk);
      const typename M::frag a1 = lds_row_frag_pad<E, D>(kt, 32 + (lane & 31), kk);
#pragma unroll
      for (int gq = 0; gq < G; ++gq) {
        s[0][gq] = M::mma(a0, qf[gq][kk], s[0][gq]);
        s[1][gq] = M::mma(a1, qf[gq][kk], s[1][gq]);
      }
    }
  };
  // Sub-tile state: 0 = nothing valid, 1 = all valid, 2 = per-element masking.
  auto sub_kind = [&](int j0, int gq) {
    const int r0 = q0 + 32 * gq, r1 = min(n - 1, r0 + 31);
    if (r0 >= n || j0 >= n || (a.causal && j0 > r1)) return 0;
    if (j0 + 31 >= n || (a.causal && j0 + 31 > r0)) return 2;
    return 1;
  };
  // Invalid keys of a masked sub-tile become -inf: never the maximum, and
  // the clamp of [x - tau]_+ makes them exactly 0.
  auto mask_tile = [&](f32x16& s, int j0, int gq) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = j0 + crow(r);
      if (!(j < n && (!a.causal || j <= qi[gq]))) s[r] = -INFINITY;
    }
  };
  // The block's sub-tiles, scored and masked; returns the kinds (k[h][gq]),
  // or false when the wave has nothing valid in the block.
  auto block = [&](int kb, const E* kt, f32x16 (&s)[2][G], int (&k)[2][G]) {
    const int j0 = kb * BLK;
    bool anyv = false, all1 = true;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int gq = 0; gq < G; ++gq) {
        k[h][gq] = sub_kind(j0 + 32 * h, gq);
        anyv |= k[h][gq] != 0;
        all1 &= k[h][gq] == 1;
      }
    if (!anyv) return false;
    scores(kt, s);
    if (!all1) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int gq = 0; gq < G; ++gq)
          if (k[h][gq] == 2) mask_tile(s[h][gq], j0 + 32 * h, gq);
    }
    return true;
  };

  // ---- pass 0: row maxima and the top-eight bound of each row (see
  // tau_solve_kernel): each lane keeps, per group, the four largest maxima of
  // its 16-score sub-tile columns.
  //
  // With a cache slot, the same pass collects the candidate lists: every
  // score above the running value of the bound.  Sub-tile maxima only grow,
  // so the running bound never exceeds the final one, and a list holds every
  // score above the final lower end of the bracket, which no later tau goes
  // below.  A wave whose lists come near their capacity filters them by the
  // current bound; if that frees too little, the workgroup stops collecting
  // and its evaluations stream K.
  float t4[G][4];
#pragma unroll
  for (int gq = 0; gq < G; ++gq)
#pragma unroll
    for (int j = 0; j < 4; ++j) t4[gq][j] = -INFINITY;
  float kj[8];  // j^(-1/gamma)
#pragma unroll
  for (int j = 0; j < 8; ++j) kj[j] = j == 0 ? 1.f : exp2f(-__log2f((float)(j + 1)) / g);
  // The maxima of the four quads of a sub-tile (scores r0 .. r0 + 3), and
  // of the sub-tile from them.
  auto quad_maxima = [&](const f32x16& s, float (&gm)[4]) {
#pragma unroll
    for (int r0 = 0; r0 < 16; r0 += 4)
      gm[r0 / 4] = max3f(s[r0], s[r0 + 1], max3f(s[r0 + 2], s[r0 + 3], s[r0 + 3]));
    return max3f(gm[0], gm[1], max3f(gm[2], gm[3], gm[3]));
  };
  // Inserts a sub-tile maximum into t4[gq].
  auto insert_max = [&](float v, int gq) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float h = fmaxf(t4[gq][j], v);
      v = fminf(t4[gq][j], v);
      t4[gq][j] = h;
    }
  };
  auto tile_max = [&](const f32x16& s, int gq) {
    float gm[4];
    insert_max(quad_maxima(s, gm), gq);
  };
  // The row's eight largest sub-tile maxima, descending: the two lanes'
  // sorted lists merged by Batcher's odd-even network (the same result in
  // both lanes of the row).
  auto row_top8 = [&](int gq, float* u) {
#pragma unroll
    for (int j = 0; j < 4; ++j) wave_halves(t4[gq][j], u[j], u[4 + j]);
    auto cx = [&](int x, int y) {
      const float hv = fmaxf(u[x], u[y]);
      u[y] = fminf(u[x], u[y]);
      u[x] = hv;
    };
    cx(0, 4); cx(1, 5); cx(2, 6); cx(3, 7);
    cx(2, 4); cx(3, 5);
    cx(1, 2); cx(3, 4); cx(5, 6);
  };
  // Lower end of the bracket (x units) from the row's eight largest
  // sub-tile maxima u (descending, distinct keys).  One term of f at a time
  // gives tau >= c u_j - j^(-1/gamma); then two Newton steps on f restricted
  // to these eight scores.  For gamma >= 1 that restricted f is convex and
  // decreasing, so Newton steps from a point below its root stay below it,
  // and its root is itself below tau (the dropped terms of f are >= 0).
  // Every z here is at most 1, as the per-element maps assume, and z_1 > 0
  // keeps the derivative nonzero.
  auto x_bound = [&](const float* u, bool refine) {
    float b = -INFINITY;
#pragma unroll
    for (int j = 0; j < 8; ++j) b = fmaxf(b, fmaf(c, u[j], -kj[j]));
    if (refine && newton_bound && b > -INFINITY) {
#pragma unroll
      for (int it = 0; it < 2; ++it) {
        float f = -1.f, fp = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float z = fmaf(c, u[j], -b);
          if (z > 0.f) {
            float pj, uj;
            Gamma<GK>::pu(z, g, pj, uj);
            f += pj;
            fp += uj;
          }
        }
        b += f / (g * fp);
      }
    }
    return b;
  };
  // the bound in score units, less a margin that covers the rounding of
  // x = c s and of the bound itself (a superset of entries is harmless)
  auto score_bound = [&](const float* u, bool refine) {
    const float b = x_bound(u, refine) / c;
    return b - 1e-5f * fmaxf(fabsf(b), 1.f / c);
  };

  int cc[G] = {};    // entries (quads, or singles of a later fill) in this thread's two lists
  int cmax[G] = {};  // wave maxima of cc once the cache is in use
  int ns[G] = {};    // compacted singles in this thread's two lists
  int nsmax[G] = {}; // their wave maxima
  // index of quad e of list gq of this thread
  constexpr uint32_t ENTRY_STEP = G * SV_NT;
  auto entry_idx = [&](int e, int gq) {
    return (uint32_t)e * ENTRY_STEP + (uint32_t)(gq * SV_NT + (int)threadIdx.x);
  };
  // Stores a quad and its key at index idx (32-bit byte offsets from the
  // workgroup-uniform array bases need no 64-bit address arithmetic).
  auto put = [&](uint32_t idx, const f32x4& v, int key4) {
    *reinterpret_cast<f32x4*>(slot + idx * 16u) = v;
    *reinterpret_cast<uint16_t*>(kslot + idx * 2u) = (uint16_t)key4;
  };
  // the scores r0 .. r0 + 3 of a sub-tile (keys crow(r0) .. crow(r0) + 3)
  auto quad_of = [](const f32x16& t, int r0) {
    return f32x4{t[r0], t[r0 + 1], t[r0 + 2], t[r0 + 3]};
  };
  auto max4 = [](const f32x4& v) { return fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])); };
  auto wave_max = [&](int v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = max(v, __shfl_xor(v, o));
    return v;
  };
  auto max_over = [](const int (&v)[G]) {
    int m = v[0];
#pragma unroll
    for (int gq = 1; gq < G; ++gq) m = max(m, v[gq]);
    return m;
  };
  // whether v[gq] > limit for some group
  auto any_over = [](const int (&v)[G], int limit) {
    bool r = false;
#pragma unroll
    for (int gq = 0; gq < G; ++gq) r |= v[gq] > limit;
    return r;
  };
  // Loads of list entries through buffer resources over the slot's arrays:
  // a lane past its own count gets an offset past the end of the resource,
  // so that nothing is fetched for it (the value, 0, is never used).  The
  // scans below run the wave's longest list, so this saves the reads of
  // the shorter ones.
  const uint32_t qbytes = (uint32_t)a.cap * G * SV_NT * 16;
  const __amdgpu_buffer_rsrc_t rq = buffer_rsrc(slot, qbytes), rkq = buffer_rsrc(kslot, qbytes / 8),
                               rsc = buffer_rsrc(sslot, qbytes / 4), rbk = buffer_rsrc(bslot, qbytes / 8),
                               rfl = buffer_rsrc(slot, (uint32_t)scap * G * SV_NT * 8);
  auto off_if = [&](bool ok, int e, int gq, uint32_t size) { return ok ? entry_idx(e, gq) * size : BUFFER_OOB; };
  auto ld_quad = [&](int e, int gq, bool ok) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rq, off_if(ok, e, gq, 16u), 0, 0));
  };
  auto ld_qkey = [&](int e, int gq, bool ok) {
    return (int)__builtin_amdgcn_raw_buffer_load_b16(rkq, off_if(ok, e, gq, 2u), 0, 0);
  };
  auto ld_single = [&](int e, int gq, bool ok) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsc, off_if(ok, e, gq, 4u), 0, 0));
  };
  auto ld_block = [&](int e, int gq, bool ok) {
    return (int)__builtin_amdgcn_raw_buffer_load_b16(rbk, off_if(ok, e, gq, 2u), 0, 0);
  };
  auto ld_fill = [&](int e, int gq, bool ok) {
    return __builtin_bit_cast(CandEntry, __builtin_amdgcn_raw_buffer_load_b64(rfl, off_if(ok, e, gq, 8u), 0, 0));
  };
  // Reads list gq of this thread in batches of eight independent quad
  // loads, up to the wave's longest list cmax rounded up to a multiple of 8
  // (inside the slot: cmax <= cap, and cap is a multiple of 8).
  // use(quad, key) for each quad of list gq.
  auto scan_quads = [&](int gq, auto&& use) {
    for (int e0 = 0; e0 < cmax[gq]; e0 += 8) {
      f32x4 qv[8];
      int kv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool ok = e0 + u < cc[gq];
        qv[u] = ld_quad(e0 + u, gq, ok);
        kv[u] = ld_qkey(e0 + u, gq, ok);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (e0 + u < cc[gq]) use(qv[u], kv[u]);
    }
  };
  // The scores of both lists for an evaluation: eight quads from each list
  // per batch, up to the longer wave maximum rounded up to 8.  use(gq, score)
  // in list order.
  auto scan_scores = [&](auto&& use) {
    const int m = max_over(cmax);
    for (int e0 = 0; e0 < m; e0 += 8) {
      f32x4 v[G][8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int gq = 0; gq < G; ++gq) v[gq][u] = ld_quad(e0 + u, gq, e0 + u < cc[gq]);
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int gq = 0; gq < G; ++gq)
          if (e0 + u < cc[gq]) {
#pragma unroll
            for (int i = 0; i < 4; ++i) use(gq, v[gq][u][i]);
          }
    }
  };
  // The compacted singles of both lists for an evaluation (4-byte loads).
  auto scan_scores_compact = [&](auto&& use) {
    const int m = max_over(nsmax);
    for (int e0 = 0; e0 < m; e0 += 8) {
      float v[G][8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int gq = 0; gq < G; ++gq) v[gq][u] = ld_single(e0 + u, gq, e0 + u < ns[gq]);
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int gq = 0; gq < G; ++gq)
          if (e0 + u < ns[gq]) use(gq, v[gq][u]);
    }
  };
  // The compacted singles of list gq with their key blocks: use(score, kb).
  auto scan_compact = [&](int gq, auto&& use) {
    for (int e0 = 0; e0 < nsmax[gq]; e0 += 8) {
      float v[8];
      int kv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool ok = e0 + u < ns[gq];
        v[u] = ld_single(e0 + u, gq, ok);
        kv[u] = ld_block(e0 + u, gq, ok);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (e0 + u < ns[gq]) use(v[u], kv[u]);
    }
  };
  // The quads of both lists with their keys: use(gq, quad, key).
  auto scan_quads_both = [&](auto&& use) {
    const int m = max_over(cmax);
    for (int e0 = 0; e0 < m; e0 += 8) {
      f32x4 v[G][8];
      int kq[G][8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int gq = 0; gq < G; ++gq) {
          const bool ok = e0 + u < cc[gq];
          v[gq][u] = ld_quad(e0 + u, gq, ok);
          kq[gq][u] = ld_qkey(e0 + u, gq, ok);
        }
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int gq = 0; gq < G; ++gq)
          if (e0 + u < cc[gq]) use(gq, v[gq][u], kq[gq][u]);
    }
  };
  // Lists of singles of a later fill: use(score, key).
  auto scan_singles = [&](int gq, auto&& use) {
    for (int e0 = 0; e0 < cmax[gq]; e0 += 8) {
      CandEntry ce[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) ce[u] = ld_fill(e0 + u, gq, e0 + u < cc[gq]);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (e0 + u < cc[gq]) use(ce[u].s, ce[u].j);
    }
  };
  auto scan_scores_singles = [&](auto&& use) {
    const int m = max_over(cmax);
    for (int e0 = 0; e0 < m; e0 += 8) {
      float v[G][8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int gq = 0; gq < G; ++gq) v[gq][u] = ld_fill(e0 + u, gq, e0 + u < cc[gq]).s;
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int gq = 0; gq < G; ++gq)
          if (e0 + u < cc[gq]) use(gq, v[gq][u]);
    }
  };
  // Keeps the quads of list gq with a score above `sb` (all lanes of the
  // wave).  In place: a quad moves only to a position already read.
  auto filter = [&](int gq, float sbv) {
    cmax[gq] = wave_max(cc[gq]);
    int k = 0;
    scan_quads(gq, [&](const f32x4& v, int key4) {
      if (max4(v) > sbv) put(entry_idx(k++, gq), v, key4);
    });
    cc[gq] = k;
  };
  float sb[G];  // collection thresholds
#pragma unroll
  for (int gq = 0; gq < G; ++gq) sb[gq] = -INFINITY;
  __shared__ int fill_dead;              // a list overflowed: stop collecting
  if (threadIdx.x == 0) fill_dead = 0;   // read after the first block's barrier
  // With a cache slot, a first stream over the leading key blocks finds
  // their sub-tile maxima, so that the collection below starts from a bound
  // close to its final value instead of collecting (and later dropping) most
  // scores of its first blocks.  Those blocks' maxima are then not inserted
  // again (the bound needs distinct keys).  The stream covers an eighth of
  // the key blocks, half of them, or all of them.  After the eighth it
  // counts the threads holding a score of the last block above the bound of
  // the maxima so far, and stops there if at most WARM_STOP of them do: for
  // rows with few large scores the collection is cheap and a longer stream
  // only adds MFMA work, for rows with many it saves list stores.  At d = 64,
  // where a block's products cost half as much against the collection work
  // they save, more than WARM_ALL such threads take the stream over every
  // block (B8 H12 n1024 c = 1: 0.120 against 0.153 ms; where fewer pass,
  // half was faster, e.g. B4 H12 n4096 causal c = 8 0.195 against 0.213 ms
  // for every block).  (Measured at n = 8192 with a
  // fixed length: an eighth, a quarter and a half of the blocks cost 0.77 /
  // 0.75 / 0.73 ms at c = 1, while at c = 16 and at n = 65536 causal the
  // eighth was the fastest.  The count after an eighth is 189 of 256
  // threads at c = 1, 95 at c = 2, 49 at c = 4 and 23 at c = 16.)
  int W = 0;
  if (cache) {
    const int w_lo = max(1, nkb / 8);
    int w_hi = max(1, nkb / 2);
    dma.issue(kbuf[0], K, 0, n);
    for (int kb = 0;; ++kb) {
      dma_wait();
      __syncthreads();
      if (kb + 1 < w_hi) dma.issue(kbuf[(kb + 1) & 1], K, (kb + 1) * BLK, n);
      f32x16 s[2][G];
      int k[2][G];
      const bool valid = block(kb, kbuf[kb & 1], s, k);
      if (valid) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int gq = 0; gq < G; ++gq)
            if (k[h][gq]) tile_max(s[h][gq], gq);
      }
      W = kb + 1;
      if (W >= w_hi) break;
      if (W == w_lo) {
        int above = 0;
#pragma unroll
        for (int gq = 0; gq < G; ++gq) {
          float u[8];
          row_top8(gq, u);
          const float b = row_ok[gq] ? score_bound(u, true) : INFINITY;
          if (valid) {
#pragma unroll
            for (int h = 0; h < 2; ++h)
              if (k[h][gq]) {
#pragma unroll
                for (int r = 0; r < 16; ++r) above += s[h][gq][r] > b ? 1 : 0;
              }
          }
        }
        const int cnt = __syncthreads_count(above > 0);
        if (cnt <= WARM_STOP) break;
        if (D <= 64 && cnt > WARM_ALL) w_hi = nkb;
      }
    }
    dma_wait();  // the copy of block W may still be in flight
    __syncthreads();
#pragma unroll
    for (int gq = 0; gq < G; ++gq) {
      float u[8];
      row_top8(gq, u);
      sb[gq] = row_ok[gq] ? score_bound(u, true) : INFINITY;
    }
  }
  // The collection starts after the first stream's blocks, whose maxima are
  // in, and takes them last, at the bound of all the others: fewer of their
  // scores pass than at the bound of the first stream alone.
  stream_from(W < nkb ? W : 0, [&](int kb, const E* kt) {
    // once the lists have overflowed, the first stream's blocks need nothing
    // more (their maxima are in)
    if (kb < W && fill_dead) return;
    f32x16 s[2][G];
    int k[2][G];
    if (!block(kb, kt, s, k)) return;
    float tm[2][G], gm[2][G][4];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int gq = 0; gq < G; ++gq) {
        const float v = quad_maxima(s[h][gq], gm[h][gq]);
        tm[h][gq] = k[h][gq] ? v : -INFINITY;
        if (kb >= W && k[h][gq]) insert_max(v, gq);
      }
    if (!cache || fill_dead) return;
    // Every 4 blocks the running bound takes the one-term bound of the
    // current maxima, every 32 blocks the Newton-refined one (any valid
    // lower bound serves; the first stream already left a close one).  The
    // maxima only change from block W on.
    if (kb >= W && (kb & 3) == 0) {
#pragma unroll
      for (int gq = 0; gq < G; ++gq) {
        float u[8];
        row_top8(gq, u);
        if (row_ok[gq]) sb[gq] = fmaxf(sb[gq], score_bound(u, (kb & 31) == 0));
      }
    }
    // a block adds at most 8 quads to each list
#pragma unroll
    for (int gq = 0; gq < G; ++gq) {
      if (__ballot(cc[gq] > a.cap - 8) != 0ull) {
        filter(gq, sb[gq]);
        if (__ballot(cc[gq] > a.cap - 8) != 0ull) {
          fill_dead = 1;
          return;
        }
      }
    }
    // Only sub-tiles whose maximum passes in some lane are searched; in them
    // each lane appends the quads holding a score above the bound, with one
    // 16-byte store per quad instead of one store per score.  The scores of
    // a quad below the bound are 0 at every tau of the bracket, as in a
    // streamed pass.  The quads keep the stream's order.
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int gq = 0; gq < G; ++gq)
        if (__ballot(tm[h][gq] > sb[gq]) != 0ull) {
#pragma unroll
          for (int r0 = 0; r0 < 16; r0 += 4) {
            if (gm[h][gq][r0 / 4] > sb[gq]) {
              put(entry_idx(cc[gq], gq), quad_of(s[h][gq], r0), (kb * BLK + 32 * h + crow(r0)) >> 2);
              ++cc[gq];
            }
          }
        }
  });

  float lo[G], hi[G], tau[G];
#pragma unroll
  for (int gq = 0; gq < G; ++gq) {
    float u[8];
    row_top8(gq, u);
    lo[gq] = hi[gq] = tau[gq] = 0.f;
    if (row_ok[gq]) {
      const float m = c * u[0];
      hi[gq] = m - powf((float)ni[gq], 1.f - a.alpha);
      const float b = x_bound(u, true);
      // the bound may round above the root by a few ulps (rows whose whole
      // support is among the eight reach it)
      lo[gq] = fminf(b - 4e-6f * fmaxf(1.f, fabsf(b)), hi[gq]);
      tau[gq] = 0.5f * (lo[gq] + hi[gq]);
    }
  }

  int passes = 1;  // K passes (streamed), the max pass included
  int evals = 0;   // evaluations of f, f', f'' (Algorithm 1 iterations)
  // Evaluations run on the lists when every one of them fit.  Entries below
  // the final bound (collected while it was still rising) stay: at any tau
  // of the bracket their z is clamped to exactly 0, as in a streamed pass.
  bool cached = cache && !__syncthreads_or(fill_dead != 0);
  if (cached) {
#pragma unroll
    for (int gq = 0; gq < G; ++gq) cmax[gq] = wave_max(cc[gq]);
  }
  int attempts = cache ? 1 : 0;  // cache fills tried (pass 0 is the first)
  // form of the lists: 0 quads, 1 compacted singles, 2 singles of a later fill
  int lists = 0;
  bool fits = false;             // a fill at the current lower end would fit
  float f_prev[G];
#pragma unroll
  for (int gq = 0; gq < G; ++gq) f_prev[gq] = INFINITY;

  for (int it = 0;; ++it) {
    // ---- evaluation at tau (per group): m0 = sum z^gamma, m1 = sum
    // z^(gamma-1), m2 = sum z^(gamma-2) over the strict support z > 0, mc =
    // the size of the support.
    float m0[G] = {}, m1[G] = {}, m2[G] = {};
    int mc[G] = {};
    auto add_z = [&](float zp, int gq) {
      if constexpr (GK == 1) {
        m0[gq] += zp;
        mc[gq] += in_support(zp);
      } else if constexpr (GK == 2) {
        m0[gq] = fmaf(zp, zp, m0[gq]);
        m1[gq] += zp;
        mc[gq] += in_support(zp);
      } else if constexpr (GK == 4) {
        const float z2 = zp * zp;
        m0[gq] = fmaf(z2, z2, m0[gq]);
        m1[gq] = fmaf(z2, zp, m1[gq]);
        m2[gq] += z2;
        mc[gq] += in_support(zp);
      } else {
        if (zp > 0.f) {
          const float l = __log2f(zp);
          m0[gq] += exp2f(g * l);
          m1[gq] += exp2f((g - 1.f) * l);
          m2[gq] += exp2f((g - 2.f) * l);
          ++mc[gq];
        }
      }
    };
    // Adds one sub-tile; returns whether it holds a positive probability.
    auto eval_tile = [&](const f32x16& s, int gq) {
      if constexpr (GK == 1 || GK == 2) {
        int cnt = 0;
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float za = relu_z(c, s[r], tau[gq]), zb = relu_z(c, s[r + 1], tau[gq]);
          if constexpr (GK == 1) {
            m0[gq] += za;
            m0[gq] += zb;
          } else {
            m0[gq] = fmaf(za, za, m0[gq]);
            m0[gq] = fmaf(zb, zb, m0[gq]);
            m1[gq] += za;
            m1[gq] += zb;
          }
          cnt += in_support(za) + in_support(zb);
        }
        mc[gq] += cnt;
        return cnt > 0;
      } else {
        bool any = false;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float zp = relu_z(c, s[r], tau[gq]);
          any |= zp > 0.f;
          add_z(zp, gq);
        }
        return any;
      }
    };
    // Appends the entries x > lo of a sub-tile to list gq; every later tau
    // stays >= lo, so entries left out are 0 there.  The threshold in score
    // units carries a margin for the rounding of lo / c.
    float s_lo[G];
#pragma unroll
    for (int gq = 0; gq < G; ++gq) {
      const float t0 = lo[gq] / c;
      s_lo[gq] = row_ok[gq] ? t0 - 1e-6f * fmaxf(fabsf(t0), 1.f / c) : INFINITY;
    }
    // (this fill stores single scores: after an evaluation the bracket is
    // narrow and few scores of a quad are above its lower end)
    auto fill_tile = [&](const f32x16& s, int gq, int jb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (s[r] > s_lo[gq]) {
          if (cc[gq] < scap)
            *reinterpret_cast<CandEntry*>(slot + entry_idx(cc[gq], gq) * 8u) = CandEntry{s[r], jb + crow(r)};
          ++cc[gq];
        }
      }
    };
    auto fill_done = [&]() {
      if (!__syncthreads_or(any_over(cc, scap))) {
        cached = true;
        lists = 2;
#pragma unroll
        for (int gq = 0; gq < G; ++gq) cmax[gq] = wave_max(cc[gq]);
      }
    };

    // If the lists of pass 0 overflowed, collecting them is tried once more
    // in a K pass of its own, when the first streamed evaluation counted few
    // enough scores above its lower end: the fill keeps the scores above the
    // lower end as it stands now, which has only risen since, so it fits.
    if (!cached && cache && it >= 1 && attempts < 2 && fits) {
      ++attempts;
#pragma unroll
      for (int gq = 0; gq < G; ++gq) cc[gq] = 0;
      stream([&](int kb, const E* kt) {
        f32x16 s[2][G];
        int k[2][G];
        if (!block(kb, kt, s, k)) return;
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int gq = 0; gq < G; ++gq)
            if (k[h][gq]) fill_tile(s[h][gq], gq, kb * BLK + 32 * h);
      });
      ++passes;
      fill_done();
    }
    if (!cached) {
      // streamed evaluation; the mask bits of every block are rewritten.  The
      // first one after an overflow also counts the scores above the lower
      // end, the size of a fill at this point.
      const bool count = cache && attempts < 2;
      int over[G] = {};
      // with G = 1 two waves share the words of a query block, so they are
      // cleared here and each wave ORs its bits in (after the stream's first
      // barrier)
      if constexpr (G == 1)
        for (int x = lane; x < TW; x += 64) bits[qbl * BW + x] = 0;
      uint32_t word = 0;  // mask bits of the current 32-block group (wave-uniform)
      stream([&](int kb, const E* kt) {
        f32x16 s[2][G];
        int k[2][G];
        bool any = false;
        if (block(kb, kt, s, k)) {
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int gq = 0; gq < G; ++gq)
              if (k[h][gq]) {
                any |= eval_tile(s[h][gq], gq);
                if (count) {
#pragma unroll
                  for (int r = 0; r < 16; ++r) over[gq] += s[h][gq][r] > s_lo[gq] ? 1 : 0;
                }
              }
        }
        if (__ballot(any) != 0ull) word |= 1u << (kb & 31);
        if ((kb & 31) == 31 || kb == nkb - 1) {
          if (lane == 0) {
            if constexpr (G == 2)
              bits[qbl * BW + (kb >> 5)] = word;
            else
              atomicOr(&bits[qbl * BW + (kb >> 5)], word);
          }
          word = 0;
        }
      });
      ++passes;
      if (count) {
        fits = !__syncthreads_or(any_over(over, scap));
        if (!fits) attempts = 2;  // no retry, and no more counting
      }
    } else if (lists == 2) {
      scan_scores_singles([&](int gq, float sv) { add_z(relu_z(c, sv, tau[gq]), gq); });
    } else if (lists == 1) {
      scan_scores_compact([&](int gq, float sv) { add_z(relu_z(c, sv, tau[gq]), gq); });
    } else if (it == 0) {
      // first evaluation on the quads: also copies the scores above the
      // lower end (every later tau stays >= lo, so the others are 0 there)
      // into the compacted lists, in the same order
      // Each score is stored unconditionally through buffer resources that
      // end with the compacted arrays: a score that stays out, or one past
      // the capacity, gets an offset past the end and its stores are
      // dropped (no branches, one increment of the count).
      int cs[G] = {};
      const uint32_t sbytes = (uint32_t)a.cap * G * SV_NT * 4;
      const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(sslot, sbytes), rk = buffer_rsrc(bslot, sbytes / 2);
      scan_quads_both([&](int gq, const f32x4& v, int key4) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float x = v[i];
          add_z(relu_z(c, x, tau[gq]), gq);
          const bool keep = x > s_lo[gq];
          const uint32_t off = keep ? entry_idx(cs[gq], gq) * 4u : BUFFER_OOB;
          // (__float_as_uint of a named float: a bit cast of the vector
          // element itself stored element 0 for every i)
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), rs, off, 0, 0);
          __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(key4 >> 4), rk, off >> 1, 0, 0);
          cs[gq] += keep ? 1 : 0;
        }
      });
      if (!__syncthreads_or(any_over(cs, a.cap))) {
        lists = 1;
#pragma unroll
        for (int gq = 0; gq < G; ++gq) {
          ns[gq] = cs[gq];
          nsmax[gq] = wave_max(ns[gq]);
        }
      }
    } else {
      scan_scores([&](int gq, float sv) { add_z(relu_z(c, sv, tau[gq]), gq); });
    }

    bool conv = true;
    float f[G], f1[G], f2[G];
#pragma unroll
    for (int gq = 0; gq < G; ++gq) {
      if constexpr (GK == 1) m1[gq] = (float)mc[gq];
      if constexpr (GK == 2) m2[gq] = (float)mc[gq];
      m0[gq] = sum_halves(m0[gq]);
      m1[gq] = sum_halves(m1[gq]);
      m2[gq] = sum_halves(m2[gq]);
      f[gq] = m0[gq] - 1.f;  // Eq. 3
      if constexpr (GK == 1) {  // Eq. 6, 7
        f1[gq] = -m1[gq];
        f2[gq] = 0.f;
      } else if constexpr (GK == 2) {
        f1[gq] = -2.f * m1[gq];
        f2[gq] = 2.f * m2[gq];
      } else if constexpr (GK == 4) {
        f1[gq] = -4.f * m1[gq];
        f2[gq] = 12.f * m2[gq];
      } else {
        f1[gq] = -g * m1[gq];
        f2[gq] = g * (g - 1.f) * m2[gq];
      }
      conv &= !row_ok[gq] || fabsf(f[gq]) <= a.tol;
    }
    // A streamed evaluation has just written the mask bits at this tau, so
    // the loop ends here.  With cached scores the bits are rebuilt at the
    // end from the returned tau, so the update from this last evaluation
    // is still taken: one more Halley step costs nothing there.
    const bool stop = __syncthreads_and(conv) || it >= a.max_iter;
    evals = it + 1;
    if (stop && !cached) break;
#pragma unroll
    for (int gq = 0; gq < G; ++gq) {
      if (!row_ok[gq]) continue;
      // the update rules of tau_solve_kernel: B_f (Eq. 4), the Newton lower
      // bound for convex f, H_f (Eq. 5) with the bracket test and slack, and
      // for gamma < 1 the midpoint when |f| has not halved
      if (f[gq] < 0.f)
        hi[gq] = tau[gq];
      else
        lo[gq] = tau[gq];
      const float slack = 1e-6f * fmaxf(1.f, fmaxf(fabsf(lo[gq]), fabsf(hi[gq])));
      if (newton_bound && f1[gq] < 0.f) {
        const float tn = tau[gq] - f[gq] / f1[gq] - 10.f * slack;
        lo[gq] = fminf(fmaxf(lo[gq], tn), hi[gq]);
      }
      const float th = tau[gq] - 2.f * f[gq] * f1[gq] / (2.f * f1[gq] * f1[gq] - f[gq] * f2[gq]);
      bool take = th >= lo[gq] - slack && th <= hi[gq] + slack;
      if (!newton_bound && fabsf(f[gq]) > 0.5f * f_prev[gq]) take = false;
      f_prev[gq] = fabsf(f[gq]);
      tau[gq] = take ? fminf(fmaxf(th, lo[gq]), hi[gq]) : 0.5f * (lo[gq] + hi[gq]);
    }
    if (stop) break;
  }

  if constexpr (precise_path<E, GK>()) {
    // ---- fp32 inputs, general alpha (ea_common.h): tau refined in fp64 and
    // written as tau + tau_lo, and the mask written at the refined tau.  Every
    // entry above the lower edge of the band is taken with its fp64 score;
    // Newton steps on f (Eq. 3, 6) from the fp32 tau, which is already close
    // to the root, square the error each time.  The result stays in the
    // bracket, widened by the rounding of its fp32 ends.
    const float* Qf = reinterpret_cast<const float*>(Q);
    const float* Kf = reinterpret_cast<const float*>(K);
    float band[G];
    double t64[G];
#pragma unroll
    for (int gq = 0; gq < G; ++gq) {
      band[gq] = PRECISE_BAND * fmaxf(1.f, fabsf(tau[gq]));
      t64[gq] = tau[gq];
    }
    // use(group, fp32 score, key) for every valid entry of this lane's rows:
    // from the lists when they hold every candidate, else from a K pass
    auto visit = [&](auto&& use) {
      if (cached && lists == 2) {
#pragma unroll
        for (int gq = 0; gq < G; ++gq) scan_singles(gq, [&](float sv, int jv) { use(gq, sv, jv); });
      } else if (cached) {
#pragma unroll
        for (int gq = 0; gq < G; ++gq)
          scan_quads(gq, [&](const f32x4& v, int key4) {
#pragma unroll
            for (int i = 0; i < 4; ++i) use(gq, v[i], 4 * key4 + i);
          });
      } else {
        stream([&](int kb, const E* kt) {
          f32x16 s[2][G];
          int k[2][G];
          if (!block(kb, kt, s, k)) return;
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int gq = 0; gq < G; ++gq)
              if (k[h][gq]) {
#pragma unroll
                for (int r = 0; r < 16; ++r) use(gq, s[h][gq][r], kb * BLK + 32 * h + crow(r));
              }
        });
        ++passes;
      }
    };
    // fp64 z of an entry, or -1 for one below the band (outside the support)
    auto z64 = [&](int gq, float sv, int jv) -> double {
      const float raw = fmaf(c, sv, -tau[gq]);
      if (!(raw > -band[gq])) return -1.0;
      return exact_x<D>(Qf + (size_t)qi[gq] * D, Kf + (size_t)jv * D, a.c64) - t64[gq];
    };
    for (int it = 0; it < 3; ++it) {
      double s0[G] = {}, s1[G] = {};
      visit([&](int gq, float sv, int jv) {
        if (!row_ok[gq]) return;
        const double z = z64(gq, sv, jv);
        if (z > 0.0) {
          s0[gq] += pow(z, a.g64);
          s1[gq] += pow(z, a.g64 - 1.0);
        }
      });
#pragma unroll
      for (int gq = 0; gq < G; ++gq) {
        s0[gq] += __shfl_xor(s0[gq], 32);
        s1[gq] += __shfl_xor(s1[gq], 32);
        if (row_ok[gq] && s1[gq] > 0.0) {
          const double slack = 1e-5 * fmax(1.0, fmax(fabs((double)lo[gq]), fabs((double)hi[gq])));
          const double tn = t64[gq] + (s0[gq] - 1.0) / (a.g64 * s1[gq]);
          t64[gq] = fmin(fmax(tn, (double)lo[gq] - slack), (double)hi[gq] + slack);
        }
      }
    }
    if (lane < 32) {
#pragma unroll
      for (int gq = 0; gq < G; ++gq)
        if (row_ok[gq]) {
          const float th = (float)t64[gq];
          a.tau[(size_t)bh * n + qi[gq]] = th;
          a.tau_lo[(size_t)bh * n + qi[gq]] = (float)(t64[gq] - (double)th);
        }
    }
    for (int x = lane; x < TW; x += 64) bits[qbl * BW + x] = 0;
    __syncthreads();
    visit([&](int gq, float sv, int jv) {
      if (!row_ok[gq]) return;
      const float raw = fmaf(c, sv, -tau[gq]);
      if (raw >= band[gq] || z64(gq, sv, jv) > 0.0) {
        const int kv = jv >> 6;
        atomicOr(&bits[qbl * BW + (kv >> 5)], 1u << (kv & 31));
      }
    });
  } else {
    if (lane < 32) {
#pragma unroll
      for (int gq = 0; gq < G; ++gq)
        if (row_ok[gq]) {
          a.tau[(size_t)bh * n + qi[gq]] = tau[gq];
          if (std::is_same<E, float>::value) a.tau_lo[(size_t)bh * n + qi[gq]] = 0.f;
        }
    }
    if (cached) {
      // mask bits at the returned tau from the cached entries
      for (int x = lane; x < TW; x += 64) bits[qbl * BW + x] = 0;
      __syncthreads();
#pragma unroll
      for (int gq = 0; gq < G; ++gq) {
        if (lists == 2) {
          scan_singles(gq, [&](float sv, int jv) {
            const int kv = jv >> 6;
            if (in_support(relu_z(c, sv, tau[gq]))) atomicOr(&bits[qbl * BW + (kv >> 5)], 1u << (kv & 31));
          });
          continue;
        }
        if (lists == 1) {
          scan_compact(gq, [&](float sv, int kv) {
            if (in_support(relu_z(c, sv, tau[gq]))) atomicOr(&bits[qbl * BW + (kv >> 5)], 1u << (kv & 31));
          });
          continue;
        }
        scan_quads(gq, [&](const f32x4& v, int key4) {
          bool any = false;
#pragma unroll
          for (int i = 0; i < 4; ++i) any |= in_support(relu_z(c, v[i], tau[gq])) != 0;
          if (any) {
            const int kv = key4 >> 4;  // key block of the quad
            atomicOr(&bits[qbl * BW + (kv >> 5)], 1u << (kv & 31));
          }
        });
      }
    }
  }
  __syncthreads();
  if (!wave_ok || !writer) return;
  // The block's mask row and its row table (Sec. 3.2.1): Q_i ascending, by
  // a ballot and a prefix count per 64 key blocks.
  int32_t* const row = a.q_index + ((size_t)bh * T + qb) * T;
  int listed = 0;
  for (int k0 = 0; k0 < T; k0 += 64) {
    const int kb = k0 + lane;
    const bool b = kb < T && ((bits[qbl * BW + (kb >> 5)] >> (kb & 31)) & 1u);
    if (kb < T) a.mask[((size_t)bh * T + qb) * T + kb] = b ? 1 : 0;
    const unsigned long long m = __ballot(b);
    if (b) row[listed + __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u))] = kb;
    listed += __popcll(m);
  }
  if (lane == 0) a.q_count[(size_t)bh * T + qb] = listed;
  if (a.stats && lane == 0) {
    a.stats[(size_t)bh * T + qb] = passes;
    a.stats[((size_t)a.BH + bh) * T + qb] = evals;
  }
}

// One workgroup per tile.  With a workspace of fewer slots than tiles the
// tiles go in launches of at most `slots` workgroups, each workgroup using
// the slot of its index, so that no two workgroups in flight share a slot
// (launches on one stream run in order).  Causal tiles come longest first,
// so each launch holds tiles of similar length.
template <typename K>
hipError_t launch_tiles(K kernel, TauArgs a, int rows, int threads, hipStream_t s) {
  const int tiles = a.BH * ((a.n + rows - 1) / rows);
  const int per = a.cand && a.slots > 0 && a.slots < tiles ? a.slots : tiles;
  for (int t0 = 0; t0 < tiles; t0 += per) {
    a.tile0 = t0;
    const hipError_t e = launch_kernel(kernel, dim3((unsigned)(tiles - t0 < per ? tiles - t0 : per)),
                                       dim3(threads), s, a);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename E, int D, int MODE>
hipError_t launch_tau_d(const TauArgs& a, hipStream_t s) {
  auto kernel = tau_solve_kernel<E, D, 0, MODE>;
  if (a.gk == 1) kernel = tau_solve_kernel<E, D, 1, MODE>;
  if (a.gk == 2) kernel = tau_solve_kernel<E, D, 2, MODE>;
  if (a.gk == 4) kernel = tau_solve_kernel<E, D, 4, MODE>;
  return launch_tiles(kernel, a, TAU_ROWS, TAU_NT, s);
}

template <typename E, int D, int G>
hipError_t launch_solve_g(TauArgs a, hipStream_t s) {
  auto kernel = solve_kernel<E, D, 0, G>;
  if (a.gk == 1) kernel = solve_kernel<E, D, 1, G>;
  if (a.gk == 2) kernel = solve_kernel<E, D, 2, G>;
  if (a.gk == 4) kernel = solve_kernel<E, D, 4, G>;
  // a slot of the two-group form holds the lists of two one-group tiles
  if (G == 1) a.slots *= 2;
  return launch_tiles(kernel, a, SV_ROWS / 2 * G, SV_NT, s);
}

// The one-group form has twice the workgroups, each wave with half the rows
// and three waves per SIMD instead of two, but every K fragment read from
// LDS feeds one product instead of two and twice as many workgroups stream
// K.  It runs grids of fewer than two 256-row tiles per compute unit, and at
// d = 64 (half the fragment reads per product) rows of up to 32768 keys.
// Measured solver times, one-group against two-group form: B8 H12 n1024 d64
// 0.122 against 0.160 ms (c = 1); B4 H12 n4096 d64 causal 0.20 against 0.25;
// B1 H8 d64 causal n = 16384 / 32768 / 65536: 0.27 / 1.14 / 4.50 against
// 0.42 / 1.21 / 4.04; B1 H16 n8192 d128: 0.75 against 0.62.
template <typename E, int D>
hipError_t launch_solve_d(const TauArgs& a, hipStream_t s) {
  const int64_t tiles = (int64_t)a.BH * ((a.n + SV_ROWS - 1) / SV_ROWS);
  if (tiles < SV_G1_BELOW || (D <= 64 && a.n <= SV_G1_MAX_N)) return launch_solve_g<E, D, 1>(a, s);
  return launch_solve_g<E, D, 2>(a, s);
}

template <int MODE>
hipError_t launch_tau_mode(const TauArgs& a, int dtype, int head_dim, hipStream_t s) {
  if (dtype == 0)
    return head_dim == 64 ? launch_tau_d<__bf16, 64, MODE>(a, s) : launch_tau_d<__bf16, 128, MODE>(a, s);
  return head_dim == 64 ? launch_tau_d<float, 64, MODE>(a, s) : launch_tau_d<float, 128, MODE>(a, s);
}

}  // namespace

hipError_t launch_tau(const TauArgs& a, int dtype, int head_dim, hipStream_t s) {
  if (dtype == 0)
    return head_dim == 64 ? launch_solve_d<__bf16, 64>(a, s) : launch_solve_d<__bf16, 128>(a, s);
  return head_dim == 64 ? launch_solve_d<float, 64>(a, s) : launch_solve_d<float, 128>(a, s);
}

hipError_t launch_tau_fused(const TauArgs& a, int dtype, int head_dim, hipStream_t s) {
  return a.o2 ? launch_tau_mode<FUSED_O2>(a, dtype, head_dim, s)
              : launch_tau_mode<FUSED_O>(a, dtype, head_dim, s);
}

}  // namespace ea
