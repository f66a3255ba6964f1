// LinSimp forward on gfx950: feature-bank preparation, chunk prefix states,
// the chunk scan with a causal log-space frame, and the anchor-window readout.
//
// Method (per head, 0-based rows; the paper counts from 1):
//   phi(x) = m^{-1/2} exp(Omega x - |x|^2/2)                  [Sec. 3.2, eq:prf]
//   M_i = sum_{j<=i} phi(k_j) v_j^T, a_i = sum_{j<=i} phi(k_j) [eq:Mstate, eq:astate]
//   z_ic = q_i (*) r_c,  C_i = {max(0,i-w+1) .. i}              [Sec. 3.2, 3.3]
//   N_i = sum_c [phi(z_ic)^T M_i] (*) u_c,  Z_i = sum_c phi(z_ic)^T a_i,
//   out_i = N_i / (Z_i + eps)                                   [eq:Ni, eq:Zi, eq:linearized-output]
//
// Everything is evaluated in log2 space.  Query side (App. B.2): one shift
// L_i = max over valid (c, p) of the log features, kept online across anchor
// tiles and feature blocks.  Key side: a causal running maximum R_j of the key
// log features; key features are exp2(lambda_j - R_j)/sqrt(m) and every state
// carries its frame, so neither side can overflow and a row never sees a
// future token's scale.  The 1/sqrt(m) of the query feature is dropped (it
// cancels in the ratio, App. A "Feature scaling").
#include <type_traits>

#include "common.h"
#include "linsimp_internal.h"
#include "prof.h"
#include "keyfeat.h"

namespace linsimp {

struct FwdArgs {
  const void* q; const void* k; const void* v; const void* r; const void* u;
  const float* omega;
  void* out; float* stats;
  void* omq; void* omk; void* omh;
  float* states; float* rho; float* rex;
  void* states16;     // [BH][nch][m][Dv] bf16 inputs: the boundary states' M in bf16; null for float32
  float* final_M; float* final_a; float* final_rex;   // optional state after the last token
  float* part;                                        // [NFB][BH][n][Dv+2] when m > 128
  void* chi;          // [BH][n][m] key features 2^(lambda_j - R_j)/sqrt(m), p permuted in 16-blocks
  float* rj;          // [BH][n]    running key frame R_j (log2)
  int H; int n; int w; int nch; int BH; float eps;
};

// ---------------------------------------------------------------------------
// K0: Omega * log2(e) in the operand type; key side keeps a hi/lo bf16 split so
// that key log features are accurate to ~2^-16 relative (bf16 keys are exact).
// bf16 inputs also get an f16 copy for the query-side logits (f16 matrix cores).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_prep_omega(const float* __restrict__ omega, T* __restrict__ omq,
                                                    T* __restrict__ omk, f16* __restrict__ omh, int H, int MD,
                                                    int D) {
  using F = MF<T>;
  int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= H * MD) return;
  float x = omega[idx] * kLog2e;
  omq[idx] = (T)x;
  // the key-side copy in fragment order (the order of bank_frag)
  const int hh = idx / MD, e = idx % MD, p = e / D, k = e % D;
  const size_t f = ((size_t)((p >> 5) * (D / F::KS) + k / F::KS) * 64 + ((k % F::KS) / F::KPL) * 32 + (p & 31))
                   * F::KPL + k % F::KPL;
  if constexpr (sizeof(T) == 2) {
    omh[idx] = (f16)x;
    bf16 hi = (bf16)x;
    omk[(size_t)hh * 2 * MD + f] = hi;
    omk[(size_t)hh * 2 * MD + MD + f] = (bf16)(x - (float)hi);
  } else {
    omk[(size_t)hh * MD + f] = (T)x;
  }
}

// ---------------------------------------------------------------------------
// K2: per 32-token chunk b, its contribution to the prefix state in the frame
// rho_b = max key log2-feature of the chunk:
//   Mt_b = sum_j chi_j v_j^T, at_b = sum_j chi_j, chi_j = exp2(lambda_j - rho_b)/sqrt(m)
// One wave per chunk.  [App. C "Host preparation": per-chunk contributions]
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M>
__global__ __launch_bounds__(256) void k_chunk_state(FwdArgs a) {
  using F = MF<T>;
  constexpr int PAD = F::PAD;
  constexpr int S = M * DV + M;
  __shared__ __align__(16) T sVt[4][DV][32 + PAD];
  __shared__ __align__(16) float snk[4][32];
  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  const int b = blockIdx.x * 4 + wv;
  const int bh = blockIdx.y, hh = bh % a.H, n = a.n;
  const bool active = b < a.nch;
  const int tok0 = b * 32;
  const T* ks = (const T*)a.k + (size_t)bh * n * D;
  const T* vs = (const T*)a.v + (size_t)bh * n * DV;
  const T* omk_h = (const T*)a.omk + (size_t)hh * (sizeof(T) == 2 ? 2 : 1) * M * D;
  f32x16 acc[M / 32];
  float nk = 0.0f;
  if (active) {
    // V^T of the chunk, token index permuted (it pairs with a register operand):
    // every 16-byte row piece is loaded first (rows clamped), then stored transposed
    constexpr int VE = 16 / (int)sizeof(T);
    constexpr int IT = 32 * (DV / VE) / 64;
    static_assert(32 * (DV / VE) % 64 == 0, "whole pieces per lane");
    typedef T VP __attribute__((ext_vector_type(VE)));
    VP xv[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = l + 64 * it, jj = idx % 32, d0 = (idx / 32) * VE;
      xv[it] = *(const VP*)(vs + (size_t)min(tok0 + jj, n - 1) * DV + d0);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = l + 64 * it, jj = idx % 32, d0 = (idx / 32) * VE;
      const bool ok = tok0 + jj < n;
#pragma unroll
      for (int e = 0; e < VE; ++e) sVt[wv][d0 + e][F::sigma(jj)] = ok ? xv[it][e] : (T)0.0f;
    }
    key_logits<T, D, M, false>(acc, nk, ks, tok0, n, omk_h);
    if (h == 0) snk[wv][col] = nk;
  }
  __syncthreads();
  if (!active) return;
  float mx = kNegInf;
  float nkt[16];
  crow_vals(snk[wv], nkt);
#pragma unroll
  for (int pt = 0; pt < M / 32; ++pt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float x = acc[pt][v] - 0.5f * kLog2e * nkt[v];
      acc[pt][v] = (tok0 + crow(v, h) < n) ? x : kNegInf;
      mx = fmaxf(mx, acc[pt][v]);
    }
  const float rb = wave_max(mx);
  const float rs = rsqrtf((float)M);
  float* st = a.states + ((size_t)bh * a.nch + b) * S;
  // bf16 inputs: the two operands of Mt_b = chi^T V are left in the chunk's
  // (otherwise unused) float32 M slot, as the 16-byte fragments the matrix
  // cores take: chi^T [p][sigma(j)] (m x 32) and V^T [d][sigma(j)] (DV x 32);
  // k_state_scan_mma forms the product and scans it
  bf16* cx = (bf16*)st;
  bf16* vx = cx + M * 32;
#pragma unroll
  for (int pt = 0; pt < M / 32; ++pt) {
    float asum = 0.0f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float c = fast_exp2(acc[pt][v] - rb) * rs;
      acc[pt][v] = c;
      asum += c;
    }
    asum = half_swap_add(asum);
    if (h == 0) st[M * DV + pt * 32 + col] = asum;
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int sp = 0; sp < F::CSTEPS; ++sp)
        *(bf16x8*)(cx + (pt * 32 + col) * 32 + 16 * sp + 8 * h) = F::cfrag(acc[pt], sp);
    } else {
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt) {
        f32x16 o = zero16();
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp)
          o = F::mma(F::cfrag(acc[pt], sp), F::ldc(&sVt[wv][dt * 32 + col][0], 0, sp, h), o);
#pragma unroll
        for (int v = 0; v < 16; ++v) st[(size_t)(pt * 32 + crow(v, h)) * DV + dt * 32 + col] = o[v];
      }
    }
  }
  if constexpr (sizeof(T) == 2) {
    for (int idx = l; idx < DV * 4; idx += 64)
      *(bf16x8*)(vx + (idx >> 2) * 32 + 8 * (idx & 3)) = *(const bf16x8*)(&sVt[wv][idx >> 2][8 * (idx & 3)]);
  }
  if (l == 0) a.rho[(size_t)bh * a.nch + b] = rb;
}

// ---------------------------------------------------------------------------
// K2b: exclusive scan over chunks with the log-scale monoid
//   (M1, R1) + (M2, r2) = (e^{R1-R} M1 + e^{r2-R} M2, R = max(R1, r2))
// in place: chunk b's contribution is replaced by the state of every token
// before chunk b, in frame rex[b] (-inf for the empty state).  With bf16
// inputs the M part of that state goes to states16 in bf16 instead (the
// operand type of every kernel that reads it, rounded once here; half the
// bytes for the scan and its readers) and only a stays in place.
// Element-parallel, sequential over chunks, loads issued PF chunks ahead.
// [App. C "Host preparation": exclusive cumulative sum -> boundary states]
// ---------------------------------------------------------------------------
template <int M, int DV>
__global__ __launch_bounds__(256) void k_state_scan(FwdArgs a) {
  constexpr int PF = 8;
  constexpr int S = M * DV + M;
  const int bh = blockIdx.y;
  const int i4 = (blockIdx.x * 256 + threadIdx.x) * 4;
  const bool act = i4 < S;
  const int nch = a.nch;
  float* st = a.states + (size_t)bh * nch * S;
  bf16* s16 = a.states16 != nullptr ? (bf16*)a.states16 + (size_t)bh * nch * M * DV : nullptr;
  const float* rh = a.rho + (size_t)bh * nch;
  float* rx = a.rex + (size_t)bh * (nch + 1);
  const bool writer = (blockIdx.x == 0 && threadIdx.x == 0);
  f32x4 run = {0.f, 0.f, 0.f, 0.f};
  float R = kNegInf;
  for (int b0 = 0; b0 < nch; b0 += PF) {
    f32x4 x[PF];
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      if (act && b0 + e < nch) x[e] = *(const f32x4*)(st + (size_t)(b0 + e) * S + i4);
      else x[e] = run * 0.0f;
    }
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      int b = b0 + e;
      if (b >= nch) break;
      float rb = rh[b];
      float Rn = fmaxf(R, rb);
      float sa = fast_exp2(R - Rn);      // 0 when R = -inf
      float sb = fast_exp2(rb - Rn);
      if (s16 != nullptr && i4 < M * DV) {
        if (act) {
          bf16x4 y;
#pragma unroll
          for (int e = 0; e < 4; ++e) y[e] = (bf16)run[e];
          *(bf16x4*)(s16 + (size_t)b * M * DV + i4) = y;
        }
      } else if (act) {
        *(f32x4*)(st + (size_t)b * S + i4) = run;
      }
      if (writer) rx[b] = R;
      run = run * sa + x[e] * sb;
      R = Rn;
    }
  }
  if (a.final_M != nullptr && act) {
    if (i4 < M * DV) *(f32x4*)(a.final_M + (size_t)bh * M * DV + i4) = run;
    else *(f32x4*)(a.final_a + (size_t)bh * M + (i4 - M * DV)) = run;
  }
  if (writer) {
    rx[nch] = R;
    if (a.final_rex != nullptr) a.final_rex[bh] = R;
  }
}

// ---------------------------------------------------------------------------
// Key features of every token in the causal running frame (one wave per chunk,
// after the scan has fixed each chunk's entry frame Rex_b):
//   R_j = max(Rex_b, max_{s0 <= j' <= j} max_p lambda_j'p),  chi_j = 2^(lambda_j - R_j)/sqrt(m)
// stored with p permuted inside 16-blocks (the LDS operand layout), for the
// readout's intra-chunk correction and, through the shared workspace, the
// backward sweeps.
// ---------------------------------------------------------------------------
template <typename T, int D, int M>
__global__ __launch_bounds__(256) void k_keyfeat(FwdArgs a) {
  using F = MF<T>;
  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  const int bh = blockIdx.y, hh = bh % a.H, n = a.n, nch = a.nch;
  const int cb = blockIdx.x * 4 + wv;
  if (cb >= nch) return;
  const int s0 = cb * 32;
  const size_t seq = (size_t)bh * n;
  const T* ks = (const T*)a.k + seq * D;
  const T* omk_h = (const T*)a.omk + (size_t)hh * (sizeof(T) == 2 ? 2 : 1) * M * D;
  f32x16 acc[M / 32];
  float nk;
  key_logits<T, D, M, true>(acc, nk, ks, s0, n, omk_h);
  const bool vt = s0 + col < n;
  float mx = kNegInf;
#pragma unroll
  for (int pt = 0; pt < M / 32; ++pt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float x = vt ? acc[pt][v] - 0.5f * kLog2e * nk : kNegInf;
      acc[pt][v] = x;
      mx = fmaxf(mx, x);
    }
  mx = half_swap_max(mx);
  float R = mx;
#pragma unroll
  for (int o = 1; o < 32; o <<= 1) {
    float t = __shfl_up(R, o, 32);
    if (col >= o) R = fmaxf(R, t);
  }
  R = fmaxf(R, a.rex[(size_t)bh * (nch + 1) + cb]);
  if (vt && h == 0) a.rj[seq + s0 + col] = R;
  const float rsm = rsqrtf((float)M);
  // the wave's 32 x M tile goes through LDS, so that the global stores are
  // whole 16-byte pieces of rows (lanes along a row) instead of 8-byte pieces
  // of 32 different rows
  constexpr int CP = M + 16 / (int)sizeof(T);              // row pitch (elements)
  __shared__ __align__(16) T sX[4][32][CP];
  T* xr = &sX[wv][col][0];
#pragma unroll
  for (int pt = 0; pt < M / 32; ++pt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      typedef T V4 __attribute__((ext_vector_type(4)));
      V4 x4;
#pragma unroll
      for (int e = 0; e < 4; ++e) x4[e] = (T)(fast_exp2(acc[pt][4 * g + e] - R) * rsm);
      *(V4*)(xr + F::sigma(pt * 32 + 8 * g + 4 * h)) = x4;   // sigma keeps 4-groups contiguous
    }
  wave_lds_sync();
  constexpr int VE = 16 / (int)sizeof(T), PPR = M / VE;    // 16-byte pieces per row
  typedef T V __attribute__((ext_vector_type(VE)));
  T* dst = (T*)a.chi + (seq + s0) * M;
  const int nrow = min(32, n - s0);
  // every piece read from LDS first, only the stores conditional (a read under
  // the condition would be a branch that waits for it)
  constexpr int IT = 32 * PPR / 64;
  V xs[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int idx = l + 64 * it, r = idx / PPR, c = (idx % PPR) * VE;
    xs[it] = *(const V*)(&sX[wv][r][c]);
  }
  no_hoist();                                   // (and not sunk into the branches)
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int idx = l + 64 * it, r = idx / PPR, c = (idx % PPR) * VE;
    if (r < nrow) *(V*)(dst + (size_t)r * M + c) = xs[it];
  }
}

// ---------------------------------------------------------------------------
// Prefill: the state after all n tokens of each (sequence, head), directly
// (eq:Mstate, eq:astate summed over the whole prefix, Theorem 1).  One
// workgroup per (sequence, head); wave wv owns features 32 wv .. 32 wv + 31 and
// walks the chunks in order, keeping its rows of M and a in registers in the
// running key frame R (log2): per chunk, the key log2-features (bf16 hi/lo
// Omega, two MFMAs per k-step: the hi half of the wave's tile in registers,
// the lo half of all tiles in LDS, so that two workgroups fit on a CU with
// two waves per SIMD), the chunk maximum shared across the waves,
// the frame update (M, a scaled by 2^(R - R')), then M += chi^T V on the
// matrix cores.  The chunk's k rows and V^T are staged in LDS one chunk ahead,
// from registers loaded two chunks ahead.
// Nothing but the final state is written (the chunked forward materialises
// every chunk's contribution instead).  bf16 inputs, m <= 128.
// ---------------------------------------------------------------------------
template <int D, int DV, int M>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_prefill_state(FwdArgs a) {
  using T = bf16;
  using F = MF<T>;
  constexpr int PAD = F::PAD, PT = M / 32;
  static_assert(PT <= 4, "one feature tile per wave");
  __shared__ __align__(16) T sK[2][32][D + PAD];
  __shared__ __align__(16) T sOl[M][D + PAD];
  __shared__ __align__(16) T sVt[2][DV][32 + PAD];
  __shared__ __align__(16) float snk[4][32];
  __shared__ float smx[4];
  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  const int bh = blockIdx.x, hh = bh % a.H, n = a.n, nch = a.nch;
  const bool owner = wv < PT;
  const size_t seq = (size_t)bh * n;
  const T* ks = (const T*)a.k + seq * D;
  const T* vs = (const T*)a.v + seq * DV;
  const T* omk_h = (const T*)a.omk + (size_t)hh * 2 * M * D;
  // hi half of this wave's Omega tile: B operands, lanes <-> feature p
  typename F::frag oh[D / F::KS];
#pragma unroll
  for (int s = 0; s < D / F::KS; ++s) oh[s] = *(const typename F::frag*)(omk_h + bank_frag<T, D>(owner ? wv : 0, s, l));
  {
    // the lo half into LDS rows: fragment f of the bank goes to row 32 pt + col,
    // columns s KS + h KPL onwards (every load issued before the first store)
    constexpr int NS = D / F::KS, NF = (M / 32) * NS * 64, IT = (NF + 255) / 256;
    static_assert(NF * F::KPL == M * D, "one fragment per lane, k-step and tile");
    typename F::frag xs[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it)
      xs[it] = *(const typename F::frag*)(omk_h + (size_t)M * D + (size_t)min(tid + 256 * it, NF - 1) * F::KPL);
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int f = tid + 256 * it;
      if (NF % 256 != 0 && f >= NF) continue;
      const int ln = f & 63, s = (f >> 6) % NS, pt = (f >> 6) / NS;
      *(typename F::frag*)&sOl[pt * 32 + (ln & 31)][s * F::KS + (ln >> 5) * F::KPL] = xs[it];
    }
  }
  const T* olrow = &sOl[(owner ? wv : 0) * 32 + col][0];
  f32x16 Macc[DV / 32];
#pragma unroll
  for (int dt = 0; dt < DV / 32; ++dt) Macc[dt] = zero16();
  float apart = 0.0f;                          // sum over this lane's tokens of chi_p, p = 32 wv + col
  float R = kNegInf;
  const float rs = rsqrtf((float)M);

  StageRows<T, 32, D, 256> sk;
  StageRowsT<T, 32, DV, 256> sv;
  auto stage_store = [&](int b, int buf) {
    sk.store(&sK[buf][0][0], D + PAD, b * 32, 0, n, tid);
    sv.store(b * 32, 0, n, tid, [&](int jj, int d0, const typename StageRowsT<T, 32, DV, 256>::V4& x) {
#pragma unroll
      for (int e = 0; e < 4; ++e) sVt[buf][d0 + e][F::sigma(jj)] = x[e];
    });
  };
  // chunk b + 1's rows are loaded while chunk b is folded in, and chunk b + 2's
  // as soon as chunk b + 1 is in LDS: every load has about one chunk's work to land
  sk.load(ks, D, 0, 0, n, tid);
  sv.load(vs, DV, 0, 0, n, tid);
  stage_store(0, 0);
  sk.load(ks, D, 32, 0, n, tid);
  sv.load(vs, DV, 32, 0, n, tid);

#pragma unroll 1
  for (int b = 0; b < nch; ++b) {
    const int cur = b & 1;
    __syncthreads();                           // chunk b staged; the other buffer is free
    // key log2-features of the tile: regs <-> token crow(v, h), lanes <-> p
    f32x16 acc = zero16();
    float mx = kNegInf;
    if (owner) {
      // two independent accumulation chains (hi, lo), summed at the end
      f32x16 part[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) part[i] = zero16();
      float nkp = 0.0f;
      const T* krow = &sK[cur][col][0];
#pragma unroll
      for (int s = 0; s < D / F::KS; ++s) {
        const typename F::frag kf = F::ld(krow, s * F::KS + h * F::KPL);
#pragma unroll
        for (int e = 0; e < F::KPL; ++e) { const float x = fel(kf, e); nkp += x * x; }
        part[0] = F::mma(kf, oh[s], part[0]);
        part[1] = F::mma(kf, F::ld(olrow, s * F::KS + h * F::KPL), part[1]);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = part[0][v] + part[1][v];
      const float nk = half_swap_add(nkp);     // |k|^2 of token col
      if (h == 0) snk[wv][col] = nk;
      wave_lds_sync();
      float nkt[16];
      crow_vals(snk[wv], nkt);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float x = acc[v] - 0.5f * kLog2e * nkt[v];
        acc[v] = (b * 32 + crow(v, h) < n) ? x : kNegInf;
        mx = fmaxf(mx, acc[v]);
      }
      mx = wave_max(mx);
    }
    if (l == 0) smx[wv] = mx;
    if (b + 1 < nch) {
      stage_store(b + 1, cur ^ 1);
      sk.load(ks, D, (b + 2) * 32, 0, n, tid);
      sv.load(vs, DV, (b + 2) * 32, 0, n, tid);
    }
    __syncthreads();
    const float cm = fmaxf(fmaxf(smx[0], smx[1]), fmaxf(smx[2], smx[3]));
    const float Rn = fmaxf(R, cm);
    if (owner) {
      const float sa = fast_exp2(R - Rn);      // 0 while the state is empty
      if (sa != 1.0f) {
#pragma unroll
        for (int dt = 0; dt < DV / 32; ++dt) Macc[dt] *= sa;
        apart *= sa;
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float c = fast_exp2(acc[v] - Rn) * rs;
        acc[v] = c;
        apart += c;
      }
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt)
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp)
          Macc[dt] = F::mma(F::cfrag(acc, sp), F::ldc(&sVt[cur][dt * 32 + col][0], 0, sp, h), Macc[dt]);
    }
    R = Rn;
  }
  // M rows p = 32 wv + crow(v, h) (lanes <-> d), a[p], the frame
  if (owner) {
    float* Mo = a.final_M + (size_t)bh * M * DV;
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) Mo[(size_t)(wv * 32 + crow(v, h)) * DV + dt * 32 + col] = Macc[dt][v];
    const float at = half_swap_add(apart);
    if (h == 0) a.final_a[(size_t)bh * M + wv * 32 + col] = at;
  }
  if (tid == 0) a.final_rex[bh] = R;
}

// ---------------------------------------------------------------------------
// K2b for bf16 inputs: the same exclusive scan, with each chunk's contribution
// Mt_b = chi^T V formed here on the matrix cores from the operand fragments the
// chunk kernel left in the chunk's M slot (0.2 of the bytes of a float32
// contribution).  One wave per (sequence-head, 32 features, 32 columns): the
// running state tile stays in its registers, the fragments of the chunks ahead
// are loaded PF chunks in advance (they do not depend on the recurrence), and
// each chunk's boundary state is written in bf16 to states16.  The wave of the
// first 32 columns also scans a in place.  Workgroups are dealt to the eight
// XCDs in turn; the waves of one sequence-head are numbered to land on one XCD,
// so the fragments they share come through one L2.
// [App. C "Host preparation": exclusive cumulative sum -> boundary states]
// ---------------------------------------------------------------------------
template <int M, int DV>
__global__ __launch_bounds__(64) void k_state_scan_mma(FwdArgs a) {
  constexpr int S = M * DV + M;
  constexpr int NDT = DV / 32, NPD = (M / 32) * NDT;
  constexpr int PF = 6;
  // the state tile passes through LDS so that each lane stores 32 contiguous
  // bytes (16 two-byte stores per lane would take most of the memory counter
  // that the loads in flight need)
  __shared__ __align__(16) bf16 sT[32][40];
  const int l = threadIdx.x, col = l & 31, h = l >> 5;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int bh = xcd + 8 * (slot / NPD), tt = slot % NPD;
  if (bh >= a.BH) return;                              // wave-uniform
  const int p0 = (tt / NDT) * 32, d0 = (tt % NDT) * 32;
  const int nch = a.nch;
  float* stb = a.states + (size_t)bh * nch * S;
  bf16* s16 = (bf16*)a.states16 + (size_t)bh * nch * M * DV;
  const float* rh = a.rho + (size_t)bh * nch;
  float* rx = a.rex + (size_t)bh * (nch + 1);
  const bool aw = d0 == 0;                              // also scans a (lanes of half 0)
  const bool writer = p0 == 0 && d0 == 0 && l == 0;
  bf16x8 xq[PF][4];
  float aq[PF], rq[PF];
  // every load unconditional (clamped chunk index), so that the compiler's
  // memory-counter waits see PF chunks in flight
  auto fetch = [&](int b, int e) {
    const bf16* cx = (const bf16*)(stb + (size_t)b * S);
    const bf16* vx = cx + M * 32;
    xq[e][0] = *(const bf16x8*)(cx + (p0 + col) * 32 + 8 * h);
    xq[e][1] = *(const bf16x8*)(cx + (p0 + col) * 32 + 16 + 8 * h);
    xq[e][2] = *(const bf16x8*)(vx + (d0 + col) * 32 + 8 * h);
    xq[e][3] = *(const bf16x8*)(vx + (d0 + col) * 32 + 16 + 8 * h);
    aq[e] = stb[(size_t)b * S + M * DV + p0 + col];
    rq[e] = rh[b];
  };
#pragma unroll
  for (int e = 0; e < PF; ++e) fetch(min(e, nch - 1), e);
  f32x16 run = zero16();
  float runa = 0.0f, R = kNegInf;
  // chunk b from ring slot e, then slot e takes chunk b + PF
  auto step = [&](int b, int e) {
    // the state of every token before chunk b (frame R)
#pragma unroll
    for (int v = 0; v < 16; ++v) sT[crow(v, h)][col] = (bf16)run[v];
    wave_lds_sync();
    {
      const int rr = l >> 1, c0 = 16 * (l & 1);
      const bf16x8 y0 = *(const bf16x8*)&sT[rr][c0], y1 = *(const bf16x8*)&sT[rr][c0 + 8];
      bf16* o = s16 + ((size_t)b * M + p0 + rr) * DV + d0 + c0;
      *(bf16x8*)o = y0;
      *(bf16x8*)(o + 8) = y1;
    }
    if (aw) stb[(size_t)b * S + M * DV + p0 + col] = runa;   // both halves: the same value
    if (writer) rx[b] = R;
    f32x16 c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xq[e][0], xq[e][2], zero16(), 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xq[e][1], xq[e][3], c, 0, 0, 0);
    const float rb = uniform(rq[e]);
    const float Rn = fmaxf(R, rb);
    const float sa = fast_exp2(R - Rn);                // 0 when R = -inf
    const float sb = fast_exp2(rb - Rn);
#pragma unroll
    for (int v = 0; v < 16; ++v) run[v] = run[v] * sa + c[v] * sb;
    runa = runa * sa + aq[e] * sb;
    R = Rn;
    fetch(min(b + PF, nch - 1), e);
  };
  int b0 = 0;
  for (; b0 + PF <= nch; b0 += PF) {
#pragma unroll
    for (int e = 0; e < PF; ++e) step(b0 + e, e);
  }
#pragma unroll
  for (int e = 0; e < PF; ++e)
    if (b0 + e < nch) step(b0 + e, e);
  if (a.final_M != nullptr) {
#pragma unroll
    for (int v = 0; v < 16; ++v) a.final_M[((size_t)bh * M + p0 + crow(v, h)) * DV + d0 + col] = run[v];
    if (aw) a.final_a[(size_t)bh * M + p0 + col] = runa;
  }
  if (writer) {
    rx[nch] = R;
    if (a.final_rex != nullptr) a.final_rex[bh] = R;
  }
}

// ---------------------------------------------------------------------------
// K3: anchor-window readout for one chunk of 32 rows.
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M, int NW, int NA>
struct RCfg {
  static constexpr int PAD = MF<T>::PAD;
  static constexpr int BC = 32;
  static constexpr int FB = M < 128 ? M : 128;          // feature block (<= 128 as in Alg. 1)
  static constexpr int NFB = M / FB;
  static constexpr int WIN = BC + 32 * NA - 1;           // anchor rows the chunk can touch
  static constexpr int UST = ((WIN + 2) / 4) * 4 + 2;   // odd dword stride: conflict-free 2-byte column reads
  static constexpr int RPW = (BC + NW - 1) / NW;
  static constexpr int ES = sizeof(T);
  static constexpr int a16(int x) { return (x + 15) & ~15; }
  static constexpr int oOm = 0;
  static constexpr int oMt = oOm + a16(FB * (D + PAD) * ES);
  static constexpr int oA = oMt + a16(DV * (FB + PAD) * ES);
  static constexpr int oChi = oA + (sizeof(T) == 4 ? a16(M * 4) : 0);   // float32: a of the boundary
  static constexpr int oVt = oChi + a16(BC * (FB + PAD) * ES);
  static constexpr int oR = oVt + a16(DV * (BC + PAD) * ES);
  // u of the window: bf16 inputs as f16 [window row][d] (read transposed, rows
  // in crow order, then multiplied in mixed precision); float32 transposed
  // [d][window row]
  static constexpr int TPU = tr_pad<T, DV>();
  static constexpr int UBYTES = sizeof(T) == 2 ? WIN * (DV + TPU) * ES : DV * UST * ES;
  static constexpr int oUt = oR + a16(WIN * (D + PAD) * ES);
  static constexpr int oQ = oUt + a16(UBYTES);
  static constexpr int oRj = oQ + a16(BC * (D + PAD) * ES);
  // bf16: the block's slice of a as a 3-row B operand (hi, lo, zero), permuted
  static constexpr int oAz = oRj + a16(BC * 4);
  static constexpr int BYTES = oAz + (sizeof(T) == 2 ? a16(3 * (FB + PAD) * ES) : 0);
};

template <typename T, int D, int DV, int M, int NW, int NA>
__global__ __launch_bounds__(64 * NW) void k_readout(FwdArgs a) {
  using F = MF<T>;
  using C = RCfg<T, D, DV, M, NW, NA>;
  constexpr int PAD = C::PAD, FB = C::FB, WIN = C::WIN, UST = C::UST, RPW = C::RPW;
  static_assert(C::BYTES <= 160 * 1024, "readout LDS budget");
  static_assert(64 * NW >= FB, "one thread per feature of the block");
  __shared__ __align__(16) char smem[C::BYTES];
  T* sOm = (T*)(smem + C::oOm);
  T* sMt = (T*)(smem + C::oMt);
  float* sA = (float*)(smem + C::oA);
  T* sChi = (T*)(smem + C::oChi);
  T* sVt = (T*)(smem + C::oVt);
  T* sR = (T*)(smem + C::oR);
  T* sUt = (T*)(smem + C::oUt);
  T* sQ = (T*)(smem + C::oQ);
  float* sRj = (float*)(smem + C::oRj);
  T* sAz = (T*)(smem + C::oAz);

  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  constexpr int NT = 64 * NW;
  const int2 gxy = xcd_grid_xy();
  const int cb = gxy.x, bh = gxy.y, hh = bh % a.H, n = a.n, nch = a.nch;
  const int s0 = cb * 32;
  const int wb = s0 - (32 * NA - 1);
  constexpr int S = M * DV + M;
  const size_t seq = (size_t)bh * n;
  const T* qs = (const T*)a.q + seq * D;
  const T* vs = (const T*)a.v + seq * DV;
  const T* rs_ = (const T*)a.r + seq * D;
  const T* us = (const T*)a.u + seq * DV;
  const T* omq_h = (const T*)a.omq + (size_t)hh * M * D;
  const float* bst = a.states + ((size_t)bh * nch + cb) * S;
  const float Rexb = a.rex[(size_t)bh * (nch + 1) + cb];
  const bool has_bnd = cb > 0;

  // ---- prologue ----
  const int fbk = blockIdx.z;
  {
    // every global load of the prologue first, then the LDS stores; the
    // transposed copies take the row index fastest across lanes, so the
    // 2-byte LDS writes of one instruction fall in one row
    using OmT = typename std::conditional<sizeof(T) == 2, f16, T>::type;
    StageRows<OmT, FB, D, NT> so;
    StageState<FB, DV, NT, true> sm;
    StageRowsT<T, FB, DV, NT> sm16;
    StageRowsT<T, 32, DV, NT> sv;
    StageRows<T, WIN, D, NT> sr;
    typename std::conditional<sizeof(T) == 2, StageRows<T, WIN, DV, NT>, StageRowsT<T, WIN, DV, NT>>::type su;
    StageRows<T, 32, D, NT> sq;
    StageRows<T, 32, FB, NT> sc;
    if constexpr (sizeof(T) == 2) so.load((const f16*)a.omh + ((size_t)hh * M + (size_t)fbk * FB) * D, D, 0, 0, FB, tid);
    else so.load(omq_h + (size_t)fbk * FB * D, D, 0, 0, FB, tid);
    if constexpr (sizeof(T) == 2) {
      if (has_bnd) sm16.load((const T*)a.states16 + (((size_t)bh * nch + cb) * M + (size_t)fbk * FB) * DV, DV, 0, 0, FB, tid);
    } else {
      if (has_bnd) sm.load(bst + (size_t)fbk * FB * DV, tid);
    }
    sv.load(vs, DV, s0, 0, n, tid);
    sr.load(rs_, D, wb, 0, n, tid);
    su.load(us, DV, wb, 0, n, tid);
    sq.load(qs, D, s0, 0, n, tid);
    sc.load((const T*)a.chi + seq * M + fbk * FB, M, s0, 0, n, tid);   // this block's features
    const float rjv = (tid < 32) ? a.rj[seq + min(s0 + tid, n - 1)] : 0.0f;
    const float azv = (sizeof(T) == 2 && has_bnd && tid < FB) ? bst[(size_t)M * DV + fbk * FB + tid] : 0.0f;
    float av[(M + NT - 1) / NT];
#pragma unroll
    for (int k = 0; k < (M + NT - 1) / NT; ++k) {
      const int p = tid + NT * k;
      av[k] = (sizeof(T) == 4 && has_bnd && p < M) ? bst[(size_t)M * DV + p] : 0.0f;
    }
    if constexpr (sizeof(T) == 2) so.store((f16*)sOm, D + PAD, 0, 0, FB, tid);
    else so.store(sOm, D + PAD, 0, 0, FB, tid);
    if constexpr (sizeof(T) == 2) {
      sm16.store(0, 0, FB, tid, [&](int p, int d0, const typename StageRowsT<T, FB, DV, NT>::V4& x) {
#pragma unroll
        for (int e = 0; e < 4; ++e) sMt[(d0 + e) * (FB + PAD) + F::sigma(p)] = has_bnd ? x[e] : (T)0.0f;
      });
    } else {
      sm.store(tid, [&](int p, int d0, const f32x4& x) {
#pragma unroll
        for (int e = 0; e < 4; ++e) sMt[(d0 + e) * (FB + PAD) + F::sigma(p)] = has_bnd ? (T)x[e] : (T)0.0f;
      });
    }
    if constexpr (sizeof(T) == 4) {
#pragma unroll
      for (int k = 0; k < (M + NT - 1) / NT; ++k)
        if (tid + NT * k < M) sA[tid + NT * k] = av[k];
    }
    sv.store(s0, 0, n, tid, [&](int jj, int d0, const typename StageRowsT<T, 32, DV, NT>::V4& x) {
#pragma unroll
      for (int e = 0; e < 4; ++e) sVt[(d0 + e) * (32 + PAD) + F::sigma(jj)] = x[e];
    });
    if constexpr (sizeof(T) == 2) sr.store((f16*)sR, D + PAD, wb, 0, n, tid);
    else sr.store(sR, D + PAD, wb, 0, n, tid);
    if constexpr (sizeof(T) == 2) {
      su.store((f16*)sUt, DV + C::TPU, wb, 0, n, tid);      // f16: exact for bf16 in its range
    } else {
      su.store(wb, 0, n, tid, [&](int wi, int d0, const typename StageRowsT<T, WIN, DV, NT>::V4& x) {
#pragma unroll
        for (int e = 0; e < 4; ++e) sUt[(d0 + e) * UST + wi] = x[e];
      });
    }
    if constexpr (sizeof(T) == 2) sq.store((f16*)sQ, D + PAD, s0, 0, n, tid);
    else sq.store(sQ, D + PAD, s0, 0, n, tid);
    sc.store(sChi, FB + PAD, s0, 0, n, tid);
    if (tid < 32) sRj[tid] = (s0 + tid < n) ? rjv : 0.0f;
    if constexpr (sizeof(T) == 2) {
      if (tid < FB) {
        const T hi = (T)azv;
        const int ps = F::sigma(tid);
        sAz[ps] = hi;
        sAz[FB + PAD + ps] = (T)(azv - (float)hi);
        sAz[2 * (FB + PAD) + ps] = (T)0.0f;
      }
    }
  }
  __syncthreads();

  const int fb = blockIdx.z;       // feature block handled by this workgroup
#pragma unroll 1
  for (int rr = 0; rr < RPW; ++rr) {
    const int t = wv + NW * rr;
    const int i = s0 + t;
    if (t >= C::BC || i >= n) continue;
    float nacc[DV / 32];
    float zacc = 0.0f, Lrun = kNegInf;
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) nacc[dt] = 0.0f;
    const float Ri = uniform(sRj[t]);
    const float sb = uniform(has_bnd ? fast_exp2(Rexb - Ri) : 0.0f);
    // frame ratios 2^(R_j - R_i) of the registers' rows j = crow(v, h), zero for
    // j > t: all sixteen read and formed, then selected (a load under the
    // condition would be a branch per register, each waiting for its read)
    float sj[16];
    const float* sRjh = sRj + 4 * h;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 r4 = *(const f32x4*)(sRjh + 8 * g);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = fast_exp2(r4[e] - Ri);
        sj[4 * g + e] = (8 * g + 4 * h + e <= t) ? x : 0.0f;
      }
    }
    const T* qrow = sQ + t * (D + PAD);
#pragma unroll 1
    for (int an = 0; an < NA; ++an) {
      // keep the loop-invariant LDS operand reads inside the loop (hoisting
      // them all would exhaust the register file)
      no_hoist();
      const int c = i - 32 * an - col;
      const bool valid = (32 * an + col < a.w) && (c >= 0);
      const int wi = t + 32 * NA - 1 - 32 * an - col;
      const T* rrow = sR + wi * (D + PAD);
      // G1: log2 features of the composite queries, lanes <-> anchor, regs <-> p
      f32x16 accL[FB / 32];
      float nz;
      if constexpr (sizeof(T) == 2) {
        nz = logits_f16<D, FB, D + PAD>(accL, (const f16*)qrow, (const f16*)rrow, (const f16*)sOm);
      } else {
#pragma unroll
        for (int pt = 0; pt < FB / 32; ++pt) accL[pt] = zero16();
        nz = 0.0f;
#pragma unroll 2
        for (int s = 0; s < D / F::KS; ++s) {
          const int k0 = s * F::KS + h * F::KPL;
          const float p = F::ld(qrow, k0) * F::ld(rrow, k0);
          nz += p * p;
#pragma unroll
          for (int pt = 0; pt < FB / 32; ++pt)
            accL[pt] = F::mma(F::ld(sOm + (pt * 32 + col) * (D + PAD), k0), p, accL[pt]);
        }
        nz = half_swap_add(nz);
      }
      // invalid anchors: z is finite (zero-filled rows) and the bias removes them
      const float bias = valid ? -0.5f * kLog2e * nz : kNegInf;
      float tm = kNegInf;
#pragma unroll
      for (int pt = 0; pt < FB / 32; ++pt)
#pragma unroll
        for (int v = 0; v < 16; ++v) tm = fmaxf(tm, accL[pt][v]);
      tm = wave_max(valid ? tm + bias : kNegInf);
      const float Lnew = fmaxf(Lrun, tm);
      if (Lnew > Lrun) {
        const float sc = fast_exp2(Lrun - Lnew);
        zacc *= sc;
#pragma unroll
        for (int dt = 0; dt < DV / 32; ++dt) nacc[dt] *= sc;
        Lrun = Lnew;
      }
      const float off = bias - Lnew;
      float zc = 0.0f;
      // psi in place, boundary part of Z, then the operand-typed copy
      typename F::frag pf[FB / 32][F::CSTEPS];
      if constexpr (sizeof(T) == 2) {
        // bf16: the boundary part of Z (phi(z)^T a over the block's features)
        // is one more matrix product, of psi as rounded for the boundary
        // readout of N against the columns (a_hi, a_lo, 0, ...), a_hi + a_lo
        // being a to 16 significant bits; so N and Z see the same psi
#pragma unroll
        for (int pt = 0; pt < FB / 32; ++pt) {
#pragma unroll
          for (int v = 0; v < 16; ++v) accL[pt][v] = fast_exp2(accL[pt][v] + off);
#pragma unroll
          for (int sp = 0; sp < F::CSTEPS; ++sp) pf[pt][sp] = F::cfrag(accL[pt], sp);
        }
        f32x16 accZ = zero16();
        const T* zrow = sAz + min(col, 2) * (FB + PAD);
#pragma unroll
        for (int pt = 0; pt < FB / 32; ++pt)
#pragma unroll
          for (int sp = 0; sp < F::CSTEPS; ++sp)
            accZ = F::mma(pf[pt][sp], F::ldc(zrow, pt * 32, sp, h), accZ);
#pragma unroll
        for (int v = 0; v < 16; ++v) zc += accZ[v];
      } else {
        const float* sAh = sA + fb * FB + 4 * h;      // + pt*32 + 8*(v>>2) + (v&3)
#pragma unroll
        for (int pt = 0; pt < FB / 32; ++pt) {
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x4 av = *(const f32x4*)(sAh + pt * 32 + 8 * g);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float psi = fast_exp2(accL[pt][4 * g + e] + off);
              accL[pt][4 * g + e] = psi;
              zc += psi * av[e];
            }
          }
#pragma unroll
          for (int sp = 0; sp < F::CSTEPS; ++sp) pf[pt][sp] = F::cfrag(accL[pt], sp);
        }
      }
      zc *= sb;
      // intra-chunk causal correction: P^T[j, anchor] = chi_j . psi_anchor, scaled
      // by the frame ratio 2^(R_j - R_i) and masked to j <= i
      f32x16 accP = zero16();
      const T* chirow = sChi + col * (FB + PAD);
#pragma unroll
      for (int pt = 0; pt < FB / 32; ++pt)
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp)
          accP = F::mma(F::ldc(chirow, pt * 32, sp, h), pf[pt][sp], accP);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        accP[v] *= sj[v];
        zc += accP[v];
      }
      typename F::frag ppf[F::CSTEPS];
#pragma unroll
      for (int sp = 0; sp < F::CSTEPS; ++sp) ppf[sp] = F::cfrag(accP, sp);
      // per 32-wide slice of d: boundary readout + correction, then the anchor
      // combine N += A_c (*) u_c  (lanes <-> d, regs <-> anchor)
#pragma unroll 1
      for (int dt = 0; dt < DV / 32; ++dt) {
        no_hoist();
        f32x16 accA = zero16();
        if (has_bnd) {
          const T* mrow = sMt + (dt * 32 + col) * (FB + PAD);
#pragma unroll
          for (int pt = 0; pt < FB / 32; ++pt)
#pragma unroll
            for (int sp = 0; sp < F::CSTEPS; ++sp)
              accA = F::mma(pf[pt][sp], F::ldc(mrow, pt * 32, sp, h), accA);
          if (sb != 1.0f) accA *= sb;
        }
        const T* vrow = sVt + (dt * 32 + col) * (32 + PAD);
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp) accA = F::mma(ppf[sp], F::ldc(vrow, 0, sp, h), accA);
        // anchor row index crow(v,h) = 8*(v>>2) + 4h + (v&3) -> window index falls with it
        float sacc = 0.0f;
        if constexpr (sizeof(T) == 2) {
          // u of the register's anchor at this lane's d: transposed reads of rows
          // t + 32 NA - 1 - 32 an - crow, in crow order
          auto rmap = [&](int ar) { return t + 32 * NA - 1 - 32 * an - ar; };
#pragma unroll
          for (int sp = 0; sp < F::CSTEPS; ++sp) {
            const f16x8 uf = __builtin_bit_cast(f16x8, F::tld_crow_map(sUt, DV + C::TPU, sp, dt * 32, rmap));
#pragma unroll
            for (int e = 0; e < 8; ++e) sacc = __builtin_fmaf(accA[8 * sp + e], (float)uf[e], sacc);
          }
        } else {
          const T* urow = sUt + (dt * 32 + col) * UST + (t + 32 * NA - 1 - 32 * an) - 4 * h;
#pragma unroll
          for (int v = 0; v < 16; ++v) sacc += accA[v] * tof(urow[-(8 * (v >> 2) + (v & 3))]);
        }
        nacc[dt] += sacc;
      }
        zacc += zc;
    }
    // ---- row epilogue ----
    const float Z = wave_sum(zacc);
    if constexpr (C::NFB == 1) {
      const float inv = 1.0f / (Z + a.eps);
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt) {
        float N = half_swap_add(nacc[dt]);
        if (h == 0) ((T*)a.out)[(seq + i) * DV + dt * 32 + col] = (T)(N * inv);
      }
      if (l == 0 && a.stats != nullptr) {
        a.stats[(seq + i) * 2 + 0] = Lrun;
        a.stats[(seq + i) * 2 + 1] = Z;
      }
    } else {
      // partial (N, Z, L) of this feature block; merged by k_merge_blocks
      float* pr = a.part + (((size_t)fb * a.BH + bh) * n + i) * (DV + 2);
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt) {
        float N = half_swap_add(nacc[dt]);
        if (h == 0) pr[dt * 32 + col] = N;
      }
      if (l == 0) { pr[DV] = Z; pr[DV + 1] = Lrun; }
    }
  }
}

// Merge the per-feature-block partials (online-max combine of Alg. 1 across
// blocks):  L = max_b L_b,  N = sum_b 2^(L_b - L) N_b,  Z likewise.
template <typename T, int DV, int NFB>
__global__ __launch_bounds__(256) void k_merge_blocks(FwdArgs a) {
  const size_t rows = (size_t)a.BH * a.n;
  const size_t row = (size_t)blockIdx.x * (256 / 32) + (threadIdx.x >> 5);
  const int lane = threadIdx.x & 31;
  if (row >= rows) return;
  float L = kNegInf;
#pragma unroll
  for (int b = 0; b < NFB; ++b) L = fmaxf(L, a.part[((size_t)b * rows + row) * (DV + 2) + DV + 1]);
  float Z = 0.0f;
  float sc[NFB];
#pragma unroll
  for (int b = 0; b < NFB; ++b) {
    const float* pr = a.part + ((size_t)b * rows + row) * (DV + 2);
    sc[b] = fast_exp2(pr[DV + 1] - L);
    Z += sc[b] * pr[DV];
  }
  const float inv = 1.0f / (Z + a.eps);
  for (int d = lane; d < DV; d += 32) {
    float N = 0.0f;
#pragma unroll
    for (int b = 0; b < NFB; ++b) N += sc[b] * a.part[((size_t)b * rows + row) * (DV + 2) + d];
    ((T*)a.out)[row * DV + d] = (T)(N * inv);
  }
  if (lane == 0 && a.stats != nullptr) {
    a.stats[row * 2 + 0] = L;
    a.stats[row * 2 + 1] = Z;
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M, int NA>
static int run_fwd(const Shape& s, FwdArgs a, hipStream_t st) {
  // readout waves per workgroup: the workgroup's LDS fills a CU, so its wave
  // count sets the occupancy; 12 waves (three per SIMD, at most 168 registers
  // each) hide more of each row's dependent matrix-core / VALU chain than 8,
  // although four of them get two of the chunk's 32 rows instead of three
  constexpr int NW = 12;
  const int BH = (int)s.BH();
  const int nch = (int)s.nch();
  {
    int tot = (int)s.H * M * D;
    ProfScope ps("prep_omega", st);
    k_prep_omega<T><<<(tot + 255) / 256, 256, 0, st>>>(a.omega, (T*)a.omq, (T*)a.omk, (f16*)a.omh, (int)s.H, M * D, D);
  }
  if constexpr (sizeof(T) == 2 && M <= 128) {
    if (a.out == nullptr && a.final_M != nullptr) {   // prefill: the final state only
      { ProfScope ps("prefill_state", st);
      k_prefill_state<D, DV, M><<<BH, 256, 0, st>>>(a); }
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) {
        set_error("prefill launch failed: %s", hipGetErrorString(e));
        return -4;
      }
      return 0;
    }
  }
  { ProfScope ps("chunk_state", st);
  k_chunk_state<T, D, DV, M><<<dim3((nch + 3) / 4, BH), 256, 0, st>>>(a); }
  if constexpr (sizeof(T) == 2) {
    constexpr int NPD = (M / 32) * (DV / 32);
    ProfScope ps("state_scan", st);
    k_state_scan_mma<M, DV><<<(unsigned)((BH + 7) / 8 * 8 * NPD), 64, 0, st>>>(a);
  } else {
    constexpr int S = M * DV + M;
    ProfScope ps("state_scan", st);
    k_state_scan<M, DV><<<dim3((S / 4 + 255) / 256, BH), 256, 0, st>>>(a);
  }
  if (a.out != nullptr || a.final_M == nullptr) {      // not for a prefill
    ProfScope ps("keyfeat", st);
    k_keyfeat<T, D, M><<<dim3((nch + 3) / 4, BH), 256, 0, st>>>(a);
  }
  if (a.out != nullptr) {
    constexpr int NFB = RCfg<T, D, DV, M, NW, NA>::NFB;
    { ProfScope ps("fwd_readout", st);
    k_readout<T, D, DV, M, NW, NA><<<dim3(nch, BH, NFB), 64 * NW, 0, st>>>(a); }
    if constexpr (NFB > 1) {
      ProfScope ps("fwd_merge", st);
      size_t rows = (size_t)BH * s.n;
      k_merge_blocks<T, DV, NFB><<<(unsigned)((rows + 7) / 8), 256, 0, st>>>(a);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("forward launch failed: %s", hipGetErrorString(e));
    return -4;
  }
  return 0;
}

// Prefill ring: slot j mod w holds token j of the last min(n, w) tokens; the
// slots no token reaches (n < w) are zero.  16-byte pieces of the rows, every
// piece of a batch loaded (row index clamped) before the first is stored.
template <typename T>
__global__ __launch_bounds__(256) void k_ring_fill(const T* __restrict__ r, const T* __restrict__ u,
                                                   T* __restrict__ rr, T* __restrict__ ru,
                                                   int64_t* __restrict__ pos, int H, int n, int w,
                                                   int D, int DV) {
  constexpr int VE = 16 / (int)sizeof(T), NB = 8;
  typedef T V __attribute__((ext_vector_type(VE)));
  const int bh = blockIdx.x;
  const int pr = D / VE, pw = pr + DV / VE, total = w * pw;
  // the newest token j <= n - 1 with j mod w == slot (negative: none)
  auto token = [&](int slot) { return (n - 1) - (((n - 1 - slot) % w + w) % w); };
  for (int base = 0; base < total; base += 256 * NB) {
    V x[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int idx = min(base + (int)threadIdx.x + 256 * i, total - 1);
      const int slot = idx / pw, c = idx % pw;
      const size_t j = (size_t)max(token(slot), 0);
      const T* src = c < pr ? r + ((size_t)bh * n + j) * D + c * VE : u + ((size_t)bh * n + j) * DV + (c - pr) * VE;
      x[i] = *(const V*)src;
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int idx = base + (int)threadIdx.x + 256 * i;
      if (idx >= total) continue;
      const int slot = idx / pw, c = idx % pw;
      const bool ok = token(slot) >= 0;
      V y;
#pragma unroll
      for (int e = 0; e < VE; ++e) y[e] = ok ? x[i][e] : (T)0.0f;
      T* dst = c < pr ? rr + ((size_t)bh * w + slot) * D + c * VE : ru + ((size_t)bh * w + slot) * DV + (c - pr) * VE;
      *(V*)dst = y;
    }
  }
  if (threadIdx.x == 0 && bh % H == 0) pos[bh / H] = n;
}

int launch_ring_fill(const Shape& s, const void* r, const void* u, void* ring_r, void* ring_u,
                     int64_t* pos, hipStream_t st) {
  const int BH = (int)s.BH();
  const int es = s.dtype == 1 ? 2 : 4;
  if ((s.D * es) % 16 != 0 || (s.Dv * es) % 16 != 0) {
    set_error("ring fill: rows of %d and %d elements are not whole 16-byte pieces", s.D, s.Dv);
    return -2;
  }
  if (s.dtype == 1)
    k_ring_fill<bf16><<<BH, 256, 0, st>>>((const bf16*)r, (const bf16*)u, (bf16*)ring_r, (bf16*)ring_u,
                                          pos, (int)s.H, (int)s.n, s.w, s.D, s.Dv);
  else
    k_ring_fill<float><<<BH, 256, 0, st>>>((const float*)r, (const float*)u, (float*)ring_r,
                                           (float*)ring_u, pos, (int)s.H, (int)s.n, s.w, s.D, s.Dv);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("ring fill launch failed: %s", hipGetErrorString(e));
    return -4;
  }
  return 0;
}

// Supported (dtype, D = Dv, m) combinations; w <= 64, and up to 128 where
// wide_window_ok allows it.
#define LS_FWD_CASES(X)               \
  X(bf16, 32, 32, 32)                 \
  X(bf16, 64, 64, 64)                 \
  X(bf16, 64, 64, 128)                \
  X(bf16, 128, 128, 64)               \
  X(bf16, 128, 128, 128)              \
  X(bf16, 128, 128, 256)              \
  X(float, 32, 32, 32)                \
  X(float, 32, 32, 64)                \
  X(float, 64, 64, 32)                \
  X(float, 64, 64, 64)

bool fwd_combo_supported(int dtype, int D, int Dv, int m) {
#define X(T, D_, DV_, M_) \
  if (dtype == (sizeof(T) == 2 ? 1 : 0) && D == D_ && Dv == DV_ && m == M_) return true;
  LS_FWD_CASES(X)
#undef X
  return false;
}

int launch_forward(const Shape& s, const void* q, const void* k, const void* v, const void* r,
                   const void* u, const float* omega, void* out, float* stats, float* final_M,
                   float* final_a, float* final_rex, const Workspace& ws, hipStream_t st) {
  FwdArgs a;
  a.q = q; a.k = k; a.v = v; a.r = r; a.u = u; a.omega = omega;
  a.out = out; a.stats = stats;
  a.omq = ws.omq; a.omk = ws.omk; a.omh = ws.omh; a.states = ws.states; a.states16 = ws.states16; a.rho = ws.rho; a.rex = ws.rex;
  a.final_M = final_M; a.final_a = final_a; a.final_rex = final_rex;
  a.H = (int)s.H; a.n = (int)s.n; a.w = s.w; a.nch = (int)s.nch(); a.BH = (int)s.BH(); a.eps = s.eps;
  a.part = ws.part;
  a.chi = ws.chi; a.rj = ws.rj;
  const int NA = (s.w + 31) / 32;
#define X(T, D_, DV_, M_)                                                          \
  if (s.dtype == (sizeof(T) == 2 ? 1 : 0) && s.D == D_ && s.Dv == DV_ && s.m == M_) { \
    if (NA == 1) return run_fwd<T, D_, DV_, M_, 1>(s, a, st);                      \
    if (NA == 2) return run_fwd<T, D_, DV_, M_, 2>(s, a, st);                      \
    if constexpr (wide_window_ok(sizeof(T) == 2 ? 1 : 0, D_, M_, 3)) {              \
      if (NA == 3) return run_fwd<T, D_, DV_, M_, 3>(s, a, st);                    \
    }                                                                              \
    if constexpr (wide_window_ok(sizeof(T) == 2 ? 1 : 0, D_, M_, 4)) {              \
      if (NA == 4) return run_fwd<T, D_, DV_, M_, 4>(s, a, st);                    \
    }                                                                              \
  }
  LS_FWD_CASES(X)
#undef X
  set_error("unsupported shape (dtype=%d D=%d Dv=%d m=%d)", s.dtype, s.D, s.Dv, s.m);
  return -2;
}

}  // namespace linsimp
