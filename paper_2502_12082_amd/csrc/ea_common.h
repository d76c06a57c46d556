// ea_common.h -- device building blocks shared by the alpha-entmax attention
// kernels for gfx950 (CDNA4): MFMA traits for bf16 and fp32 operands, register
// fragment loaders, 64-row LDS tiles (row-major and transposed), and the
// per-element alpha-entmax maps specialised on gamma = 1/(alpha-1).
//
// Conventions used by every kernel
// --------------------------------
// * Tensors are [B*H, n, D] row-major, D in {64, 128}; blocks are 64 rows.
// * One wave owns a 32-row slab of the "resident" side of a product and
//   computes 32x32 output tiles with v_mfma_f32_32x32x16_bf16 (bf16 inputs) or
//   v_mfma_f32_32x32x2_f32 (fp32 inputs), fp32 accumulation.
// * Accumulator layout of a 32x32 tile (identical for both instructions):
//   value r (0..15) of lane l sits at row 8*(r/4) + 4*(l/32) + (r%4), column
//   l%32.  `crow(r)` returns that row for the calling lane.
// * A and B operands: lane l supplies row (A) or column (B) l%32 and the
//   k-slice [8*(l/32), 8*(l/32)+8) of a 16-wide k step (bf16), or k = l/32 of
//   a 2-wide k step (fp32).
// * Probability tiles are fed back to the MFMA straight from the accumulator
//   registers: the contraction index is permuted (the same permutation on both
//   operands), so step t of a 32-wide contraction uses accumulator values
//   [8t, 8t+8) (bf16) or value t (fp32); `perm_key` gives the contraction row
//   that a lane's slot maps to, and the transposed LDS tiles are read with the
//   same permutation.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace ea {

constexpr int BLK = 64;  // mask block edge (rows and columns)

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
// Wave index within the workgroup, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }
// Row of accumulator value r for the calling lane (see the layout note above).
__device__ __forceinline__ int crow(int r) { return 8 * (r >> 2) + 4 * (lane_id() >> 5) + (r & 3); }

// The values that lanes l % 32 and 32 + l % 32 hold in v (the two halves of
// the wave exchange with one v_permlane32_swap, no LDS round trip).
__device__ __forceinline__ void wave_halves(float v, float& lo, float& hi) {
#if defined(__HIP_DEVICE_COMPILE__)
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
#else
  lo = hi = v;
#endif
}
// v of lane l plus v of lane l ^ 32, the same value in both lanes.
__device__ __forceinline__ float sum_halves(float v) {
  float lo, hi;
  wave_halves(v, lo, hi);
  return lo + hi;
}

// max(a, b, c) in one v_max3_f32.  fmaxf chains on MFMA results also
// canonicalise each operand (one more instruction per operand); scores are
// finite or -inf, where the two agree.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Buffer resource over `bytes` bytes at p (gfx9 layout: raw byte
// addressing).  A buffer access at a byte offset >= `bytes` is dropped by the
// hardware, which turns predicated stores into unconditional ones.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)bytes, 0x00020000);
}
constexpr uint32_t BUFFER_OOB = 0x80000000u;  // an offset past every buffer here

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// ------------------------------------------------------------ MFMA traits

template <typename E>
struct Mma;

template <>
struct Mma<__bf16> {
  using frag = bf16x8;
  static constexpr int KW = 16;   // contraction width of one instruction
  static constexpr int EPL = 8;   // operand elements per lane
  __device__ __forceinline__ static f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  // A operand from accumulator values [8t, 8t+8), rounded to nearest even.
  __device__ __forceinline__ static frag pack(const float* v, int t) {
    frag f;
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = (__bf16)v[8 * t + e];
    return f;
  }
  // Two-term split v ~ hi + lo, both bf16; hi + lo carries ~16 mantissa bits.
  // Pairs are rounded together (one v_cvt_pk_bf16_f32); the fp32 values of
  // the two hi halves come back out of the packed word with one shift and
  // one mask, and the exact remainders are rounded as a second pair.
  __device__ __forceinline__ static void pack_split(const float* v, int t, frag& hi, frag& lo) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    u32x4 hw, lw;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = v[8 * t + 2 * e], b = v[8 * t + 2 * e + 1];
      const uint32_t hp = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)a, (__bf16)b});
      const float ra = a - __uint_as_float(hp << 16);
      const float rb = b - __uint_as_float(hp & 0xFFFF0000u);
      hw[e] = hp;
      lw[e] = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)ra, (__bf16)rb});
    }
    hi = __builtin_bit_cast(bf16x8, hw);
    lo = __builtin_bit_cast(bf16x8, lw);
  }
  static constexpr bool exact_operands = false;
};

template <>
struct Mma<float> {
  using frag = float;
  static constexpr int KW = 2;
  static constexpr int EPL = 1;
  __device__ __forceinline__ static f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ __forceinline__ static frag pack(const float* v, int t) { return v[t]; }
  __device__ __forceinline__ static void pack_split(const float* v, int t, frag& hi, frag& lo) {
    hi = v[t];
    lo = 0.f;
  }
  static constexpr bool exact_operands = true;  // fp32 operands need no split
};

// Steps of a 32-wide contraction fed from accumulator registers.
template <typename E>
constexpr int perm_steps() { return 32 / Mma<E>::KW; }

// Contraction row (0..31) that slot (step t, element e) of the calling lane
// holds, under the permutation described at the top of this file.
template <typename E>
__device__ __forceinline__ int perm_key(int t, int e) {
  const int h = lane_id() >> 5;
  if constexpr (Mma<E>::EPL == 8) {
    return 8 * (2 * t + (e >> 2)) + 4 * h + (e & 3);
  } else {
    return 8 * (t >> 2) + 4 * h + (t & 3);
  }
}

// ------------------------------------------------------- global fragments

// Row fragment for k step kk of row `row` of a [*, D] row-major global
// matrix: bf16 -> 8 values at k = 16kk + 8h; fp32 -> 1 value at k = 2kk + h.
// Rows outside [0, nrows) read as zero.
template <typename E, int D>
__device__ __forceinline__ typename Mma<E>::frag load_row_frag_global(const E* base, int row,
                                                                      int nrows, int kk) {
  const int h = lane_id() >> 5;
  if constexpr (Mma<E>::EPL == 8) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < nrows) v = *reinterpret_cast<const u32x4*>(base + (size_t)row * D + 16 * kk + 8 * h);
    return __builtin_bit_cast(bf16x8, v);
  } else {
    float v = 0.f;
    if (row < nrows) v = base[(size_t)row * D + 2 * kk + h];
    return v;
  }
}

// -------------------------------------------------------------- LDS tiles
//
// A 64 x D tile of a [*, D] row-major global matrix is staged in LDS
// row-major in 16-byte chunks, chunk (r, c) of tile row r stored at chunk
// position r * CPR + (c ^ swz(r)) (CPR chunks per row).  The XOR pattern
// spreads both access patterns over the banks: 32 lanes reading one chunk
// column of 32 rows (MFMA row fragments), and the 8-row x 32-column blocks
// read by the transposing loads.
//
// Tiles are filled with global_load_lds (16 bytes per lane, written to LDS
// without passing through registers): wave instruction k writes chunk
// positions [64k, 64k + 64), so each lane fetches the global chunk whose
// swizzled position it owns.  Rows past the end of the matrix repeat its
// last row; every kernel masks those rows' contributions to exactly zero.
// Completion is awaited with dma_wait() followed by a workgroup barrier.

template <typename E, int D>
struct Tile {
  static constexpr int VEC = 16 / (int)sizeof(E);  // elements per 16-byte chunk
  static constexpr int CPR = D / VEC;              // chunks per row
  static constexpr int CHUNKS = BLK * CPR;
  static constexpr int ELEMS = BLK * D;
  // Chunk XOR pattern of tile row r, a bijection on the rows of each
  // 16-row group (32 lanes reading one chunk column hit distinct banks);
  // with 16 chunks per row the low two row bits also move whole 4-chunk
  // groups, and with 8 chunks per row (two rows per 64 banks) row r and
  // r + 2 differ in chunk bit 2, so the 4-row x 4-chunk blocks of a
  // transposing read spread over all 64 banks.
  __device__ __forceinline__ static int swz(int r) {
    if constexpr (CPR == 16) {
      return ((r & 3) << 2) | ((r >> 2) & 3);
    } else if constexpr (CPR == 8) {
      const int k = (r >> 1) & 7;
      return ((k & 1) << 2) | (k >> 1);
    } else {
      return r & (CPR - 1);
    }
  }
  __device__ __forceinline__ static int chunk_pos(int r, int c) { return r * CPR + (c ^ swz(r)); }
  // element offset of (row r, column col)
  __device__ __forceinline__ static int elem(int r, int col) {
    return chunk_pos(r, col / VEC) * VEC + (col & (VEC - 1));
  }
  // global element offset (within the 64-row block) of the chunk stored at
  // chunk position p
  __device__ __forceinline__ static int src_off(int p) {
    const int r = p / CPR;
    return r * D + ((p % CPR) ^ swz(r)) * VEC;
  }
};

// A 64 x D tile read only as MFMA row fragments, stored row-major with one
// 16-byte pad chunk after every row (row stride CPR + 1 chunks).  The 16
// rows read by 16 consecutive lanes then start in 16 distinct 16-byte bank
// groups (CPR + 1 is odd), so row-fragment reads are conflict-free, and the
// chunk offset of k step kk is the same constant for every lane: the reads
// of one row use one base address plus immediate offsets.  The pad chunks
// are filled with a copy of the row's first chunk and never read.
template <typename E, int D>
struct PadTile {
  static constexpr int VEC = 16 / (int)sizeof(E);
  static constexpr int CPR = D / VEC;
  static constexpr int RS = CPR + 1;  // row stride in chunks
  static constexpr int CHUNKS = BLK * RS;
  static constexpr int ELEMS = CHUNKS * VEC;
  __device__ __forceinline__ static int chunk_pos(int r, int c) { return r * RS + c; }
  __device__ __forceinline__ static int elem(int r, int col) {
    return chunk_pos(r, col / VEC) * VEC + (col & (VEC - 1));
  }
  __device__ __forceinline__ static int src_off(int p) {
    const int r = p / RS, c = p % RS;
    return r * D + (c == CPR ? 0 : c) * VEC;
  }
};

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

__device__ __forceinline__ lds_void_t* to_lds(const void* p) {
  return (lds_void_t*)((__attribute__((address_space(3))) char*)(p));
}

// Asynchronous copy of tile rows [row0, row0 + 64) of g ([nrows, D]) into
// an LDS tile of layout TL, spread over the NT threads of the workgroup:
// wave instruction k (k = i * NW + wave) fills chunk positions
// [64k, 64k + 64).  The element offset of every chunk this lane fetches is
// computed once (init); a copy is then one uniform base plus those offsets,
// with the row clamp only on the last, partial tile.
template <typename TL, int D, int NT>
struct TileDma {
  static constexpr int NW = NT / 64;
  static constexpr int NI = TL::CHUNKS / 64;        // wave instructions per tile
  static constexpr int PER = (NI + NW - 1) / NW;    // per wave (the last may be idle)
  static_assert(TL::CHUNKS % 64 == 0, "tile chunks must fill whole wave instructions");
  int off[PER];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < PER; ++i) off[i] = TL::src_off(64 * min(i * NW + wave_id(), NI - 1) + lane_id());
  }

  template <typename E>
  __device__ __forceinline__ void issue(E* tile, const E* g, int row0, int nrows) const {
#if defined(__HIP_DEVICE_COMPILE__)  // gfx950 builtin; kernels' lambdas are also parsed for the host
    const E* base = g + (size_t)row0 * D;
    if (row0 + BLK <= nrows) {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int k = i * NW + wave_id();
        if (NI % NW != 0 && k >= NI) break;
        __builtin_amdgcn_global_load_lds(base + off[i], to_lds(tile + 64 * k * TL::VEC), 16, 0, 0);
      }
    } else {
      const int last = nrows - 1 - row0;  // rows past the end repeat the last row
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int k = i * NW + wave_id();
        if (NI % NW != 0 && k >= NI) break;
        const int r = off[i] / D;
        const int o = off[i] + (min(r, last) - r) * D;
        __builtin_amdgcn_global_load_lds(base + o, to_lds(tile + 64 * k * TL::VEC), 16, 0, 0);
      }
    }
#endif
  }
};

template <typename E, int D, int NT>
using DmaPlan = TileDma<Tile<E, D>, D, NT>;

// Waits for this wave's outstanding global loads, global_load_lds included
// (s_waitcnt vmcnt(0)); follow with a barrier before reading the tiles.
__device__ __forceinline__ void dma_wait() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// A-operand row fragment of tile row r, k step kk.
template <typename E, int D>
__device__ __forceinline__ typename Mma<E>::frag lds_row_frag(const E* tile, int r, int kk) {
  using TL = Tile<E, D>;
  const int h = lane_id() >> 5;
  if constexpr (Mma<E>::EPL == 8) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(tile + TL::chunk_pos(r, 2 * kk + h) * 8));
  } else {
    return tile[TL::elem(r, 2 * kk + h)];
  }
}

// A-operand row fragment of row r, k step kk, of a PadTile.
template <typename E, int D>
__device__ __forceinline__ typename Mma<E>::frag lds_row_frag_pad(const E* tile, int r, int kk) {
  using TL = PadTile<E, D>;
  const int h = lane_id() >> 5;
  if constexpr (Mma<E>::EPL == 8) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(tile + TL::chunk_pos(r, 2 * kk + h) * 8));
  } else {
    return tile[TL::elem(r, 2 * kk + h)];
  }
}

// B-operand fragment for the permuted contraction over tile rows
// [rbase, rbase + 32), output column cbase + l % 32, step t.  bf16: two
// transposing reads (ds_read_b64_tr_b16): in each 16-lane group, lane j
// addresses row r0 + j/4, columns 4 (j % 4) .. +3 of a 16-column strip, and
// lane i receives column i of the four rows r0 .. r0 + 3.
template <typename E, int D>
__device__ __forceinline__ typename Mma<E>::frag lds_perm_frag(const E* tile, int cbase, int rbase, int t) {
  using TL = Tile<E, D>;
  const int l = lane_id();
  if constexpr (Mma<E>::EPL == 8) {
#if defined(__HIP_DEVICE_COMPILE__)
    const int r0 = rbase + 16 * t + 4 * (l >> 5) + ((l & 15) >> 2);
    const int col = cbase + 16 * ((l >> 4) & 1) + 4 * (l & 3);
    const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)to_lds(tile + TL::elem(r0, col)));
    const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)to_lds(tile + TL::elem(r0 + 8, col)));
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 v = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    return __builtin_bit_cast(bf16x8, v);
#else
    return bf16x8{};
#endif
  } else {
    return tile[TL::elem(rbase + perm_key<E>(t, 0), cbase + (l & 31))];
  }
}

// ------------------------------------------------- per-element entmax maps
//
// zp = clamp(x - tau, 0, 1) where x = c * s; within the bracket of Algorithm 1
// (tau >= max_j x_j - 1) every z = x - tau is <= 1, so the clamp is exactly
// [z]_+ and folds into one v_fma_f32 with the clamp bit.
__device__ __forceinline__ float relu_z(float c, float s, float tau) {
  return __builtin_amdgcn_fmed3f(fmaf(c, s, -tau), 0.f, 1.f);
}

// 1 if zp > 0, else 0, for zp from the clamp above (+0, -0 or positive; -0
// has the sign bit set and reads as a negative integer): one v_med3_i32.
__device__ __forceinline__ int in_support(float zp) {
#if defined(__HIP_DEVICE_COMPILE__)
  int r;
  asm("v_med3_i32 %0, %1, 0, 1" : "=v"(r) : "v"(zp));
  return r;
#else
  return zp > 0.f ? 1 : 0;
#endif
}

// ------------------------------------- fp32 inputs with a general alpha
//
// For gamma = 1/(alpha-1) below 2 (alpha > 1.5) u = z^(gamma-1) has an
// unbounded slope as z -> 0+ (Sec. 3.2.2, App. A.2).  An fp32 score carries
// a rounding error of ~1e-7 |x| from its fp32 accumulation, and u of an entry
// that close to the support edge can then be off by far more than the fp32
// tolerance; tau solved on fp32 scores moves the whole edge by as much.  With
// fp32 inputs and a general alpha the kernels therefore take z = x - tau in
// fp64 for every entry within PRECISE_BAND * max(1, |tau|) of the edge: the
// products of fp32 inputs are exact in fp64, and tau carries a low part
// (tau + tau_lo) that the solver refines in fp64.
template <typename E, int GK>
constexpr bool precise_path() {
  return std::is_same<E, float>::value && GK == 0;
}
constexpr float PRECISE_BAND = 0.01f;

// (alpha-1) * scale * <q, k> in fp64 for fp32 rows q, k of length D (16-byte
// aligned); every product is exact in fp64.
template <int D>
__device__ __forceinline__ double exact_x(const float* q, const float* k, double c64) {
  double a0 = 0.0, a1 = 0.0;
#pragma unroll 4
  for (int t = 0; t < D; t += 4) {
    const f32x4 x = *reinterpret_cast<const f32x4*>(q + t);
    const f32x4 y = *reinterpret_cast<const f32x4*>(k + t);
    a0 = fma((double)x[0], (double)y[0], a0);
    a1 = fma((double)x[1], (double)y[1], a1);
    a0 = fma((double)x[2], (double)y[2], a0);
    a1 = fma((double)x[3], (double)y[3], a1);
  }
  return c64 * (a0 + a1);
}

// [x - tau]_+ clamped to [0, 1] (as relu_z) for a valid entry of row q and
// key k with fp32 score s: within the band of the edge from fp64 x and the
// fp64 tau64 = tau + tau_lo, elsewhere in fp32.  `ok` is false for rows past
// the end (nothing is read then).
template <int D>
__device__ __forceinline__ float precise_relu_z(bool ok, float c, float s, float tau, float band,
                                                double tau64, const float* q, const float* k,
                                                double c64) {
  const float raw = fmaf(c, s, -tau);
  if (ok && fabsf(raw) < band) {
    const double z = exact_x<D>(q, k, c64) - tau64;
    return (float)fmin(fmax(z, 0.0), 1.0);
  }
  return __builtin_amdgcn_fmed3f(raw, 0.f, 1.f);
}

// GK = gamma for the integer cases 1 (alpha = 2), 2 (alpha = 1.5),
// 4 (alpha = 1.25); GK = 0 is any alpha > 1 via exp2/log2.
template <int GK>
struct Gamma {
  // p = zp^gamma and u = zp^(gamma-1) on the strict support zp > 0.
  __device__ __forceinline__ static void pu(float zp, float g, float& p, float& u) {
    if constexpr (GK == 1) {
      p = zp;
      u = zp > 0.f ? 1.f : 0.f;
    } else if constexpr (GK == 2) {
      p = zp * zp;
      u = zp;
    } else if constexpr (GK == 4) {
      const float z2 = zp * zp;
      u = z2 * zp;
      p = z2 * z2;
    } else {
      const float l = __log2f(zp);
      p = zp > 0.f ? exp2f(g * l) : 0.f;
      u = zp > 0.f ? exp2f((g - 1.f) * l) : 0.f;
    }
  }
  __device__ __forceinline__ static float p_only(float zp, float g) {
    if constexpr (GK == 1) {
      return zp;
    } else if constexpr (GK == 2) {
      return zp * zp;
    } else if constexpr (GK == 4) {
      const float z2 = zp * zp;
      return z2 * z2;
    } else {
      return zp > 0.f ? exp2f(g * __log2f(zp)) : 0.f;
    }
  }
};

}  // namespace ea
