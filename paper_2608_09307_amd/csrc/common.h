// Shared device helpers for the LinSimp HIP kernels (gfx950 / CDNA4).
//
// Matrix-core conventions used everywhere (wave64, 32x32 MFMA tiles):
//   lane l: col = l & 31, half h = l >> 5.
//   Operand fragment of k-step s (A or B): lane holds KPL consecutive k values
//     k = s*KS + h*KPL + e,  e = 0..KPL-1          ("natural" order)
//     bf16: v_mfma_f32_32x32x16_bf16, KS = 16, KPL = 8
//     f32 : v_mfma_f32_32x32x2_f32,   KS = 2,  KPL = 1
//   Accumulator (C/D) register v = 0..15 of a 32x32 tile holds
//     row = 8*(v>>2) + 4*h + (v&3),  col = l & 31.
//   A tile whose rows are a contraction index can be fed straight back to the
//   next MFMA as an operand (its columns become that operand's M or N index):
//   k-step s' of the 32-row tile uses registers 8s'..8s'+7 (bf16) or s' (f32),
//   i.e. tile rows crow(s', h, e).  The other operand of such an MFMA is read
//   from LDS with the same permutation: for bf16 it is stored permuted
//   (sigma swaps the 4-groups 1 and 2 of each 16-block) so that those rows
//   are one contiguous 16-byte read; for f32 it is indexed directly.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16;
typedef f16 f16x8 __attribute__((ext_vector_type(8)));
typedef f16 f16x4 __attribute__((ext_vector_type(4)));
typedef f16 f16x2 __attribute__((ext_vector_type(2)));

#define LS_DEV __device__ __forceinline__

static constexpr float kLog2e = 1.4426950408889634f;
static constexpr float kNegInf = -__builtin_inff();

LS_DEV int lane_id() { return threadIdx.x & 63; }

// Workgroups are dealt to the eight XCDs in turn by linear id (x fastest, then
// y).  This maps the (x, y) grid so that each XCD gets one contiguous run of it
// (runs of x for a fixed y first): neighbouring tiles, which stage the same
// rows, then share one L2.  A bijection when gridDim.x * gridDim.y is a
// multiple of 8; the plain order otherwise.
LS_DEV int2 xcd_grid_xy() {
  const int gx = (int)gridDim.x, nxy = gx * (int)gridDim.y;
  const int lin = (int)blockIdx.x + gx * (int)blockIdx.y;
  if (nxy % 8 != 0) return int2{(int)blockIdx.x, (int)blockIdx.y};
  const int v = (lin & 7) * (nxy >> 3) + (lin >> 3);
  return int2{v % gx, v / gx};
}

template <typename T> struct MF;

template <> struct MF<bf16> {
  static constexpr int KS = 16;      // k per instruction
  static constexpr int KPL = 8;      // k per lane
  static constexpr int PAD = 8;      // LDS row padding (elements) = 16 bytes
  typedef bf16x8 frag;
  LS_DEV static f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  LS_DEV static frag zero() { frag z; for (int e = 0; e < 8; ++e) z[e] = (bf16)0.0f; return z; }
  // natural fragment at row + k0 (k0 = s*KS + h*KPL)
  LS_DEV static frag ld(const bf16* row, int k0) { return *(const frag*)(row + k0); }
  // fragment of tile rows crow(s', h, *) from a permuted-storage row
  LS_DEV static frag ldc(const bf16* row, int base, int sp, int h) {
    return *(const frag*)(row + base + 16 * sp + 8 * h);
  }
  // C-derived fragment: registers 8s'..8s'+7 of an accumulator, scaled
  LS_DEV static frag cfrag(const f32x16& acc, int sp) {
    frag f;
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = (bf16)acc[8 * sp + e];
    return f;
  }
  static constexpr int CSTEPS = 2;   // k-steps per 32-row C tile
  // ---- fragments from K-major storage mat[k][n] (n contiguous), column n0 + (lane & 31) ----
  // natural k order: rows kbase + 8h + 0..7
  LS_DEV static frag tld_nat(const bf16* mat, int ld, int kbase, int n0);
  // crow order of k-step sp of a C-derived partner: rows kbase + 16sp + 8(e>>2) + 4h + (e&3)
  LS_DEV static frag tld_crow(const bf16* mat, int ld, int kbase, int sp, int n0);
  // crow order with an arbitrary logical-row -> storage-row map (ring buffers)
  template <class RowMap> LS_DEV static frag tld_crow_map(const bf16* mat, int ld, int sp, int n0, RowMap rm);
  // storage position of contraction index k for permuted operands
  LS_DEV static int sigma(int k) {
    int g = (k >> 2) & 3;
    int gs = (g == 1) ? 2 : (g == 2) ? 1 : g;
    return (k & ~15) | (gs << 2) | (k & 3);
  }
};

template <> struct MF<float> {
  static constexpr int KS = 2;
  static constexpr int KPL = 1;
  static constexpr int PAD = 1;
  typedef float frag;
  LS_DEV static f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  LS_DEV static frag zero() { return 0.0f; }
  LS_DEV static frag ld(const float* row, int k0) { return row[k0]; }
  LS_DEV static frag ldc(const float* row, int base, int sp, int h) {
    return row[base + 8 * (sp >> 2) + 4 * h + (sp & 3)];
  }
  LS_DEV static frag cfrag(const f32x16& acc, int sp) { return acc[sp]; }
  static constexpr int CSTEPS = 16;
  LS_DEV static frag tld_nat(const float* mat, int ld, int kbase, int n0) {
    const int l = threadIdx.x & 63;
    return mat[(kbase + (l >> 5)) * ld + n0 + (l & 31)];
  }
  LS_DEV static frag tld_crow(const float* mat, int ld, int kbase, int sp, int n0) {
    const int l = threadIdx.x & 63;
    return mat[(kbase + 8 * (sp >> 2) + 4 * (l >> 5) + (sp & 3)) * ld + n0 + (l & 31)];
  }
  template <class RowMap> LS_DEV static frag tld_crow_map(const float* mat, int ld, int sp, int n0, RowMap rm) {
    const int l = threadIdx.x & 63;
    return mat[rm(8 * (sp >> 2) + 4 * (l >> 5) + (sp & 3)) * ld + n0 + (l & 31)];
  }
  LS_DEV static int sigma(int k) { return k; }
};

// ---- transposing LDS reads (ds_read_b64_tr_b16) ----
// Within each 16-lane group, lane i receives column i of the 4 x 16 block whose
// row j is the 64-bit chunk addressed by lane 4j + i/4 (element i%4).  With
// lane L = 16*g + s addressing row k0 + (s>>2) and columns
// n0 + 16*(g&1) + 4*(s&3) of a row-major [k][n] matrix, lane L receives
// M[k0 .. k0+3][n0 + (L & 31)]: an MFMA operand fragment read from storage
// whose contiguous axis is the operand's M/N index.
typedef short s16x4 __attribute__((ext_vector_type(4)));
LS_DEV bf16x4 lds_tr4(const bf16* p) {
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  s16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
  return __builtin_bit_cast(bf16x4, r);
}
// address of this lane's 64-bit chunk for rows k0..k0+3 of a [k][n] matrix
LS_DEV const bf16* tr_addr(const bf16* mat, int ld, int k0, int n0) {
  const int L = threadIdx.x & 63, g = L >> 4, s = L & 15;
  return mat + (k0 + (s >> 2)) * ld + n0 + 16 * (g & 1) + 4 * (s & 3);
}
LS_DEV bf16x8 cat44(bf16x4 a, bf16x4 b) {
  bf16x8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
  r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
  return r;
}

LS_DEV bf16x8 MF<bf16>::tld_nat(const bf16* mat, int ld, int kbase, int n0) {
  const int h = (threadIdx.x & 63) >> 5;
  return cat44(lds_tr4(tr_addr(mat, ld, kbase + 8 * h, n0)), lds_tr4(tr_addr(mat, ld, kbase + 8 * h + 4, n0)));
}
LS_DEV bf16x8 MF<bf16>::tld_crow(const bf16* mat, int ld, int kbase, int sp, int n0) {
  const int h = (threadIdx.x & 63) >> 5;
  return cat44(lds_tr4(tr_addr(mat, ld, kbase + 16 * sp + 4 * h, n0)),
               lds_tr4(tr_addr(mat, ld, kbase + 16 * sp + 8 + 4 * h, n0)));
}
template <class RowMap>
LS_DEV bf16x8 MF<bf16>::tld_crow_map(const bf16* mat, int ld, int sp, int n0, RowMap rm) {
  const int L = threadIdx.x & 63, g = L >> 4, s = L & 15, h = L >> 5;
  const int col = n0 + 16 * (g & 1) + 4 * (s & 3);
  bf16x4 a = lds_tr4(mat + rm(16 * sp + 4 * h + (s >> 2)) * ld + col);
  bf16x4 b = lds_tr4(mat + rm(16 * sp + 8 + 4 * h + (s >> 2)) * ld + col);
  return cat44(a, b);
}

// Row padding (elements) of LDS buffers read with ds_read_b64_tr_b16.  One
// transposing read touches 8 rows x 64 bytes; it runs at full rate when the
// row pitch is 64 or 192 bytes modulo 256 (the four rows of each 16-lane group
// 16 dwords apart), e.g. 320-byte rows for 128 bf16 columns, against a half
// rate at 288 bytes and a third at 272 (measured on gfx950).  16-byte row
// reads run at the same rate for any of these pitches.
template <typename T, int N> constexpr int tr_pad() {
  if (sizeof(T) != 2) return 1;
  for (int p = 0; p < 128; p += 8) {
    const int b = (2 * (N + p)) % 256;
    if (b == 64 || b == 192) return p;
  }
  return 8;
}

// row index of accumulator register v in a 32x32 tile
LS_DEV int crow(int v, int h) { return 8 * (v >> 2) + 4 * h + (v & 3); }

// x[v] = row[crow(v, h)] for the 16 registers of an accumulator, from a
// 16-byte aligned 32-entry LDS row, as four 16-byte reads (read in full, so
// that a caller's per-register condition selects after the read instead of
// guarding it: a guarded read becomes a branch that waits for it)
LS_DEV void crow_vals(const float* row, float (&x)[16]) {
  const int h = lane_id() >> 5;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const f32x4 r4 = *(const f32x4*)(row + 8 * g + 4 * h);
#pragma unroll
    for (int e = 0; e < 4; ++e) x[4 * g + e] = r4[e];
  }
}

LS_DEV f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

template <typename T> LS_DEV float tof(T x) { return (float)x; }
template <typename T> LS_DEV T fromf(float x) { return (T)x; }

// fragment element access as float
LS_DEV float fel(const bf16x8& f, int e) { return (float)f[e]; }
LS_DEV float fel(const float& f, int) { return f; }
LS_DEV float fel(const f16x8& f, int e) { return (float)f[e]; }

LS_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// acc + the eight elements of a bf16 fragment, as rounded (pairwise dot
// products with ones: four instructions instead of eight conversions and adds)
typedef bf16 bf16x2 __attribute__((ext_vector_type(2)));
LS_DEV float add_elems(const bf16x8& f, float acc) {
  const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
  for (int e = 0; e < 8; e += 2) acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{f[e], f[e + 1]}, one, acc, false);
  return acc;
}
LS_DEV float add_elems(const float& f, float acc) { return acc + f; }

// value known to be equal in every lane -> scalar register (uniform branches)
LS_DEV float uniform(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}
LS_DEV int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// LDS writes by some lanes of a wave, then reads by other lanes of that wave
LS_DEV void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// compiler-only barrier: memory reads after it cannot be hoisted above it
LS_DEV void no_hoist() { asm volatile("" ::: "memory"); }

// ---- wave reductions (64 lanes) ----
// DPP within each 16-lane row, then the four row results are read into scalar
// registers: the result is wave-uniform and lives in an SGPR.
template <int CTRL> LS_DEV float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(x), __float_as_int(x), CTRL, 0xF, 0xF, false));
}
LS_DEV float rlane(float x, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l)); }
LS_DEV float wave_max(float x) {
  x = fmaxf(x, dpp<0xB1>(x));     // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp<0x4E>(x));     // quad_perm [2,3,0,1]
  x = fmaxf(x, dpp<0x124>(x));    // row_ror:4
  x = fmaxf(x, dpp<0x128>(x));    // row_ror:8
  return fmaxf(fmaxf(rlane(x, 0), rlane(x, 16)), fmaxf(rlane(x, 32), rlane(x, 48)));
}
LS_DEV float wave_sum(float x) {
  x += dpp<0xB1>(x);
  x += dpp<0x4E>(x);
  x += dpp<0x124>(x);
  x += dpp<0x128>(x);
  return (rlane(x, 0) + rlane(x, 16)) + (rlane(x, 32) + rlane(x, 48));
}
// x[l] (op) x[l ^ 32] via v_permlane32_swap
LS_DEV float half_swap_add(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
LS_DEV float half_swap_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Sixteen sums over the 32 lanes of each wave half at once (a reduce-scatter
// butterfly that halves the live registers at every step).  On return, lane
// (col, h) holds sum over the lanes col' of half h of x[col >> 1].
//   lanes 16 apart: v_permlane16_swap pairs rows 0-1 and 2-3 of the wave
//   lanes  8 apart: row_ror:8;  then row_half_mirror (l <-> 7 - l within 8),
//   quad_perm [2,3,0,1] and [1,0,3,2], each keeping the half selected by
//   lane bits 3, 2, 1.
LS_DEV float half_reduce16(const float (&x)[16]) {
  const int l = lane_id();
  float y[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x[k]), __float_as_uint(x[k + 8]), false, false);
    y[k] = __uint_as_float(r[0]) + __uint_as_float(r[1]);   // rows 0/2: x[k], rows 1/3: x[k+8]
  }
  const bool b3 = (l >> 3) & 1, b2 = (l >> 2) & 1, b1 = (l >> 1) & 1;
  float z[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) z[k] = (b3 ? y[k + 4] : y[k]) + dpp<0x128>(b3 ? y[k] : y[k + 4]);
  float u[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) u[k] = (b2 ? z[k + 2] : z[k]) + dpp<0x141>(b2 ? z[k] : z[k + 2]);
  float s = (b1 ? u[1] : u[0]) + dpp<0x4E>(b1 ? u[0] : u[1]);
  return s + dpp<0xB1>(s);
}

// ---- composite-query logits from f16 operands (bf16 inputs) ----
// q, r and Omega*log2(e) are kept in LDS as f16 (converted once per row,
// anchor window or workgroup), so z = q (*) r takes four packed f16
// multiplies per 16-wide k-step and |z|^2 four f16 dot products with float32
// accumulation; the logits use the f16 matrix-core instruction (same rate as
// bf16, with 11 mantissa bits for z).  Lanes <-> anchor (z rows from rrow),
// registers <-> feature (Omega rows pt*32 + col at row stride LD).
// Returns |z|^2 of the lane's anchor (both wave halves).
template <int D, int FB, int LD>
LS_DEV float logits_f16(f32x16 (&acc)[FB / 32], const f16* qrow, const f16* rrow, const f16* om) {
  const int l = lane_id(), col = l & 31, h = l >> 5;
  float nz = 0.0f;
  {
    const int k0 = h * 8;
    const f16x8 z = *(const f16x8*)(qrow + k0) * *(const f16x8*)(rrow + k0);
#pragma unroll
    for (int e = 0; e < 4; ++e) nz = __builtin_amdgcn_fdot2(f16x2{z[2 * e], z[2 * e + 1]}, f16x2{z[2 * e], z[2 * e + 1]}, nz, false);
#pragma unroll
    for (int pt = 0; pt < FB / 32; ++pt)
      acc[pt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(*(const f16x8*)(om + (pt * 32 + col) * LD + k0), z, zero16(), 0, 0, 0);
  }
#pragma unroll 1
  for (int s = 1; s < D / 16; ++s) {
    const int k0 = s * 16 + h * 8;
    const f16x8 z = *(const f16x8*)(qrow + k0) * *(const f16x8*)(rrow + k0);
#pragma unroll
    for (int e = 0; e < 4; ++e) nz = __builtin_amdgcn_fdot2(f16x2{z[2 * e], z[2 * e + 1]}, f16x2{z[2 * e], z[2 * e + 1]}, nz, false);
#pragma unroll
    for (int pt = 0; pt < FB / 32; ++pt)
      acc[pt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(*(const f16x8*)(om + (pt * 32 + col) * LD + k0), z, acc[pt], 0, 0, 0);
  }
  return half_swap_add(nz);
}

// crow-order operand fragment (see MF<bf16>::tld_crow) of a 16-bit matrix
// stored as f16; the transposing read moves raw 16-bit values
LS_DEV f16x8 tld_crow_f16(const f16* mat, int ld, int kbase, int sp, int n0) {
  const int h = (threadIdx.x & 63) >> 5;
  const bf16* m = (const bf16*)mat;
  return __builtin_bit_cast(f16x8, cat44(lds_tr4(tr_addr(m, ld, kbase + 16 * sp + 4 * h, n0)),
                                         lds_tr4(tr_addr(m, ld, kbase + 16 * sp + 8 + 4 * h, n0))));
}

// ---- batched global -> LDS staging ----
// A copy is split into load() (every global load of the calling thread, into
// registers) and store() (its LDS writes), so a kernel can issue the loads of
// several copies back to back and pay one memory round trip for all of them.
// Rows row0 .. row0 + ROWS - 1 of a [*, gstride] matrix are copied; rows
// outside [lo, hi) become zero (their loads read a clamped valid row).
template <typename T, int ROWS, int COLS, int NT>
struct StageRows {
  static constexpr int VE = 16 / (int)sizeof(T);
  static constexpr int CPR = COLS / VE;
  static constexpr int N = ROWS * CPR;
  static constexpr int IT = (N + NT - 1) / NT;
  static_assert(COLS % VE == 0, "16-byte pieces");
  typedef T V __attribute__((ext_vector_type(VE)));
  V x[IT];
  LS_DEV void load(const T* g, int gstride, int row0, int lo, int hi, int tid) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = min(tid + NT * it, N - 1);
      const int r = idx / CPR, c = (idx % CPR) * VE;
      const int gr = min(max(row0 + r, lo), hi - 1);
      x[it] = *(const V*)(g + (size_t)gr * gstride + c);
    }
  }
  // stores as Tout (the same type, or f16), times `scale` when converting
  template <typename Tout>
  LS_DEV void store(Tout* lds, int lstride, int row0, int lo, int hi, int tid, float scale = 1.0f) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + NT * it;
      if (N % NT != 0 && idx >= N) continue;
      const int r = idx / CPR, c = (idx % CPR) * VE;
      const bool ok = row0 + r >= lo && row0 + r < hi;
      typedef Tout VO __attribute__((ext_vector_type(VE)));
      VO y;
#pragma unroll
      for (int e = 0; e < VE; ++e) y[e] = ok ? (Tout)((float)x[it][e] * scale) : (Tout)0.0f;
      if ((lstride * (int)sizeof(Tout)) % (VE * (int)sizeof(Tout)) == 0) {
        *(VO*)(lds + r * lstride + c) = y;
      } else {
#pragma unroll
        for (int e = 0; e < VE; ++e) lds[r * lstride + c + e] = y[e];
      }
    }
  }
};

// FB x DV float32 block of a state (row stride DV), staged like StageRows.
// PFAST picks the piece order: row index fastest across lanes (for transposed
// LDS layouts) or the natural row-major order.
template <int FB, int DV, int NT, bool PFAST>
struct StageState {
  static constexpr int N = FB * (DV / 4);
  static constexpr int IT = (N + NT - 1) / NT;
  f32x4 x[IT];
  LS_DEV static void where(int idx, int& p, int& d0) {
    if (PFAST) { p = idx % FB; d0 = (idx / FB) * 4; }
    else { p = idx / (DV / 4); d0 = (idx % (DV / 4)) * 4; }
  }
  LS_DEV void load(const float* g, int tid) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      int p, d0;
      where(min(tid + NT * it, N - 1), p, d0);
      x[it] = *(const f32x4*)(g + (size_t)p * DV + d0);
    }
  }
  // put(p, d0, x): store four consecutive columns of row p
  template <class Put> LS_DEV void store(int tid, Put put) const {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + NT * it;
      if (N % NT != 0 && idx >= N) continue;
      int p, d0;
      where(idx, p, d0);
      put(p, d0, x[it]);
    }
  }
};

// Like StageRows, in 4-element pieces with the row index fastest across
// lanes, for stores into transposed LDS layouts (the 2-byte writes of one
// instruction then fall in one LDS row).  put(r, c0, x) stores the four
// values of row r, columns c0 .. c0 + 3 (zero for rows outside [lo, hi)).
template <typename T, int ROWS, int COLS, int NT>
struct StageRowsT {
  static constexpr int N = ROWS * (COLS / 4);
  static constexpr int IT = (N + NT - 1) / NT;
  typedef T V4 __attribute__((ext_vector_type(4)));
  V4 x[IT];
  LS_DEV void load(const T* g, int gstride, int row0, int lo, int hi, int tid) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = min(tid + NT * it, N - 1);
      const int r = idx % ROWS, c0 = (idx / ROWS) * 4;
      const int gr = min(max(row0 + r, lo), hi - 1);
      x[it] = *(const V4*)(g + (size_t)gr * gstride + c0);
    }
  }
  template <class Put> LS_DEV void store(int row0, int lo, int hi, int tid, Put put) const {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + NT * it;
      if (N % NT != 0 && idx >= N) continue;
      const int r = idx % ROWS, c0 = (idx / ROWS) * 4;
      const bool ok = row0 + r >= lo && row0 + r < hi;
      V4 y;
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = ok ? x[it][e] : (T)0.0f;
      put(r, c0, y);
    }
  }
};
