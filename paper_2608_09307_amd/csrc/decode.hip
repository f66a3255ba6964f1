// LinSimp autoregressive decode step on gfx950 (Theorem 1: the persistent
// state of a head is M, a and the last w anchor rows (r_c, u_c)).
//
// Per (sequence s, head h), token t = pos[s]:
//   lambda = log2-features of k_t;  R' = max(R, max_p lambda_p)
//   M <- 2^(R-R') M + chi v_t^T,  a <- 2^(R-R') a + chi,  chi = 2^(lambda - R')/sqrt(m)
//   (eq:Mstate / eq:astate in the frame R'; M_true = 2^R' M)
//   ring slot t mod w <- (r_t, u_t)
//   out = N / (Z + eps) over the min(t+1, w) most recent anchors (eq:Ni, eq:Zi)
// The readout uses the contraction order W = Psi^T U (matrix cores, sum over
// anchors), then N_d = sum_p M[p,d] W[p,d] fused with the state update, so
// every float32 state element is read once and written once.
#include "common.h"
#include "linsimp_internal.h"
#include "prof.h"

namespace linsimp {

struct DecArgs {
  const void* q; const void* k; const void* v; const void* r; const void* u;
  const float* omega;
  float* M; float* a; float* rho;
  void* ring_r; void* ring_u;
  int64_t* pos;
  void* out;
  int H; int w; float eps;
};

template <typename T, int D, int DV, int M, int NA, bool OM_LDS = true>
struct DCfg {
  static constexpr int PAD = MF<T>::PAD;
  static constexpr int W = 32 * NA;
  static constexpr int ES = sizeof(T);
  static constexpr int a16(int x) { return (x + 15) & ~15; }
  static constexpr int oOm = 0;                         // Omega * log2 e (when staged in LDS)
  static constexpr int oRr = oOm + (OM_LDS ? a16(M * (D + PAD) * ES) : 0);
  static constexpr int oUt = oRr + a16(W * (D + PAD) * ES);
  static constexpr int oQ = oUt + a16(DV * (W + PAD) * ES);
  static constexpr int oK = oQ + a16(D * 4);
  static constexpr int oV = oK + a16(D * 4);
  static constexpr int oChi = oV + a16(DV * 4);
  static constexpr int oAn = oChi + a16(M * 4);
  static constexpr int oNz = oAn + a16(M * 4);
  static constexpr int oRed = oNz + a16(W * 4);
  static constexpr int oN = oRed + a16(64 * 4);
  static constexpr int BYTES = oN + a16(4 * DV * 4);
};

// LDS staging of a ring in two phases, so that a caller issues every global
// load of its staging before the first LDS store (one memory round trip per
// call, not one per staged array).  Ring rows c < nv come from `ring`
// ([w][COLS]), row `slot` from `fresh` when it is given; rows nv .. ROWS-1
// (nv <= w: past the window, or slots that hold no token yet) are zero, so
// that a product with them needs no mask.  TRANS stores column-major with
// the row index permuted by MF<T>::sigma (the readout's anchor operand layout).
template <typename T, int ROWS, int COLS, bool TRANS>
struct RingStage {
  static constexpr int VE = 16 / sizeof(T);
  static constexpr int CPR = COLS / VE;
  static constexpr int N = ROWS * CPR;
  static constexpr int IT = (N + 255) / 256;
  typedef T V __attribute__((ext_vector_type(VE)));
  V x[IT];
  // unconditional loads (row clamped into the ring)
  LS_DEV void load(const T* ring, const T* fresh, int slot, int w, int tid) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = min(tid + 256 * it, N - 1), c = idx / CPR, e = (idx % CPR) * VE;
      const int cr = c < w ? c : w - 1;
      x[it] = *(const V*)((fresh != nullptr && cr == slot) ? fresh + e : ring + (size_t)cr * COLS + e);
    }
  }
  LS_DEV void store(T* dst, int ldst, int nv, int tid) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + 256 * it, c = idx / CPR, e = (idx % CPR) * VE;
      if (N % 256 != 0 && idx >= N) continue;
      if (c >= nv) {
#pragma unroll
        for (int k = 0; k < VE; ++k) x[it][k] = (T)0.0f;
      }
      if constexpr (TRANS) {
#pragma unroll
        for (int k = 0; k < VE; ++k) dst[(e + k) * ldst + MF<T>::sigma(c)] = x[it][k];
      } else {
#pragma unroll
        for (int k = 0; k < VE; ++k) dst[c * ldst + e + k] = x[it][k];
      }
    }
  }
};

// Omega * log2(e) of one head into LDS rows of pitch D + PAD, operand type
template <typename T, int D, int M>
LS_DEV void stage_omega(T* dst, const float* om, int tid) {
  constexpr int N = M * D / 4;
  constexpr int IT = N / 256;
  static_assert(N % 256 == 0, "Omega staging");
#pragma unroll 8
  for (int it = 0; it < IT; ++it) {
    const int idx = tid + 256 * it, p = idx / (D / 4), e = (idx % (D / 4)) * 4;
    const f32x4 x = *(const f32x4*)(om + (size_t)p * D + e);
#pragma unroll
    for (int k = 0; k < 4; ++k) dst[p * (D + MF<T>::PAD) + e + k] = (T)(x[k] * kLog2e);
  }
}

// Omega rows of one token's key GEMV held by this thread (M <= 128): feature
// p = 32 wv + col, the KPL-wide pieces at k0 = ks KS + h KPL.  Loaded apart
// from the GEMV so that a caller can issue the loads early.
template <typename T, int D>
struct KeyBankRows {
  float o[D / MF<T>::KS][MF<T>::KPL];
  LS_DEV void load(const float* om, int M, int tid) {
    using F = MF<T>;
    const int l = tid & 63, col = l & 31, h = l >> 5, wv = tid >> 6;
    const int p = wv * 32 + col;
    const float* orow = om + (size_t)(p < M ? p : 0) * D;
#pragma unroll
    for (int ks = 0; ks < D / F::KS; ++ks) {
      const int k0 = ks * F::KS + h * F::KPL;
      if constexpr (F::KPL % 4 == 0) {
#pragma unroll
        for (int e4 = 0; e4 < F::KPL; e4 += 4) {
          const f32x4 x = *(const f32x4*)(orow + k0 + e4);
#pragma unroll
          for (int e = 0; e < 4; ++e) o[ks][e4 + e] = x[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < F::KPL; ++e) o[ks][e] = orow[k0 + e];
      }
    }
  }
};

// Log2 key features of one token, lambda_p = (omega_p . k - |k|^2 / 2) log2(e),
// in float32 into lam[p] (LDS, p < M), from Omega rows already loaded
// (M <= 128).  Feature p's dot product is split over lanes l and l ^ 32, which
// take the alternate KPL-wide pieces of D that make up an MFMA operand
// fragment of row p; with FRAGS the fragments of Omega * log2(e) in the
// operand type are kept in omf[D / KS] for the query logits, so the bank is
// read once.  Returns max_p lambda_p; every thread calls it (it ends with a
// barrier).
template <typename T, int D, int M, bool FRAGS>
LS_DEV float key_log2_features_rows(const KeyBankRows<T, D>& kb, const float* sk, float* lam, float* sred,
                                    typename MF<T>::frag* omf) {
  using F = MF<T>;
  static_assert(M <= 128, "one feature row per thread");
  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = tid >> 6;
  float nk = 0.0f;
#pragma unroll
  for (int e = l; e < D; e += 64) nk += sk[e] * sk[e];
  nk = wave_sum(nk);
  float mx = kNegInf;
  const int p = wv * 32 + col;
  float acc = 0.0f;
#pragma unroll
  for (int ks = 0; ks < D / F::KS; ++ks) {
    const int k0 = ks * F::KS + h * F::KPL;
#pragma unroll
    for (int e = 0; e < F::KPL; ++e) acc += kb.o[ks][e] * sk[k0 + e];
    if constexpr (FRAGS) {
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int e = 0; e < F::KPL; ++e) omf[ks][e] = (T)(kb.o[ks][e] * kLog2e);
      } else {
        omf[ks] = kb.o[ks][0] * kLog2e;
      }
    }
  }
  acc = half_swap_add(acc);
  const float x = (acc - 0.5f * nk) * kLog2e;
  if (p < M) {
    mx = x;
    if (h == 0) lam[p] = x;
  }
  mx = wave_max(mx);
  if (l == 0) sred[wv] = mx;
  __syncthreads();
  return fmaxf(fmaxf(sred[0], sred[1]), fmaxf(sred[2], sred[3]));
}

// The same, loading the bank itself; any M (feature blocks of 128)
template <typename T, int D, int M, bool FRAGS>
LS_DEV float key_log2_features(const float* sk, const float* om, float* lam, float* sred,
                               typename MF<T>::frag* omf) {
  using F = MF<T>;
  static_assert(!FRAGS || M <= 128, "fragments for one feature tile per wave");
  if constexpr (M <= 128) {
    KeyBankRows<T, D> kb;
    kb.load(om, M, threadIdx.x);
    return key_log2_features_rows<T, D, M, FRAGS>(kb, sk, lam, sred, omf);
  } else {
    static_assert(M % 128 == 0, "whole feature blocks");
    const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = tid >> 6;
    float nk = 0.0f;
#pragma unroll
    for (int e = l; e < D; e += 64) nk += sk[e] * sk[e];
    nk = wave_sum(nk);
    float mx = kNegInf;
#pragma unroll
    for (int p0 = 0; p0 < M; p0 += 128) {
      const int p = p0 + wv * 32 + col;
      const float* orow = om + (size_t)p * D;
      float acc = 0.0f;
#pragma unroll
      for (int ks = 0; ks < D / F::KS; ++ks) {
        const int k0 = ks * F::KS + h * F::KPL;
        float o[F::KPL];
        if constexpr (F::KPL % 4 == 0) {
#pragma unroll
          for (int e4 = 0; e4 < F::KPL; e4 += 4) {
            const f32x4 x = *(const f32x4*)(orow + k0 + e4);
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e4 + e] = x[e];
          }
        } else {
#pragma unroll
          for (int e = 0; e < F::KPL; ++e) o[e] = orow[k0 + e];
        }
#pragma unroll
        for (int e = 0; e < F::KPL; ++e) acc += o[e] * sk[k0 + e];
      }
      acc = half_swap_add(acc);
      const float x = (acc - 0.5f * nk) * kLog2e;
      mx = fmaxf(mx, x);
      if (h == 0) lam[p] = x;
    }
    mx = wave_max(mx);
    if (l == 0) sred[wv] = mx;
    __syncthreads();
    return fmaxf(fmaxf(sred[0], sred[1]), fmaxf(sred[2], sred[3]));
  }
}

// z = q (*) r of one anchor at one k-step as an operand fragment (q float32
// in LDS, read in full for every lane), its |z|^2 summed into nz
template <typename T>
LS_DEV void composite_query(const float* q, const typename MF<T>::frag& rf, float& nz, typename MF<T>::frag& zf) {
  if constexpr (sizeof(T) == 2) {
    const f32x4 q0 = *(const f32x4*)q, q1 = *(const f32x4*)(q + 4);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float p = (e < 4 ? q0[e] : q1[e - 4]) * fel(rf, e);
      nz += p * p;
      zf[e] = (bf16)p;
    }
  } else {
    const float p = q[0] * rf;
    nz += p * p;
    zf = p;
  }
}

template <typename T, int D, int DV, int M, int NA>
// two waves per SIMD where the LDS allows two workgroups per CU (m <= 128)
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(M > 128 ? 1 : 2))) void k_decode(DecArgs A) {
  using F = MF<T>;
  constexpr int PT = M / 32;                  // feature tiles
  constexpr int PTW = (PT + 3) / 4;           // feature tiles per wave
  using C = DCfg<T, D, DV, M, NA, PTW != 1>;
  constexpr int PAD = C::PAD, W = C::W;
  static_assert(C::BYTES <= 160 * 1024, "decode LDS budget");
  __shared__ __align__(16) char smem[C::BYTES];
  T* sOm = (T*)(smem + C::oOm);
  T* sRr = (T*)(smem + C::oRr);
  T* sUt = (T*)(smem + C::oUt);
  float* sq = (float*)(smem + C::oQ);
  float* sk = (float*)(smem + C::oK);
  float* sv = (float*)(smem + C::oV);
  float* schi = (float*)(smem + C::oChi);
  float* san = (float*)(smem + C::oAn);
  float* snz = (float*)(smem + C::oNz);
  float* sred = (float*)(smem + C::oRed);
  float* sN = (float*)(smem + C::oN);

  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  const int sh = blockIdx.x, H = A.H, w = A.w;
  const int s = sh / H, hh = sh % H;
  const int64_t t = A.pos[s];
  const int slot = (int)(t % w);
  const int nvalid = (int)((t + 1 < w) ? t + 1 : w);
  const T* qt = (const T*)A.q + (size_t)sh * D;
  const T* kt = (const T*)A.k + (size_t)sh * D;
  const T* vt = (const T*)A.v + (size_t)sh * DV;
  const T* rt = (const T*)A.r + (size_t)sh * D;
  const T* ut = (const T*)A.u + (size_t)sh * DV;
  T* rr = (T*)A.ring_r + (size_t)sh * w * D;
  T* ru = (T*)A.ring_u + (size_t)sh * w * DV;
  const float* om = A.omega + (size_t)hh * M * D;
  float* Ms = A.M + (size_t)sh * M * DV;
  float* as = A.a + (size_t)sh * M;

  // The state rows this thread updates (feature tile pt = wv when each wave
  // owns one tile) and its entry of a are fetched first: their latency then
  // overlaps the staging, the key features and the logits.
  constexpr bool PRE = PTW == 1;
  float mreg[PRE ? DV / 32 : 1][16];
  const float a_old = tid < M ? as[tid] : 0.0f;

  // ---- the Omega rows of the key GEMV (m <= 128), then the token and both
  // rings (slot t mod w replaced by the new token): every load is issued before
  // the first LDS store, the bank's L2 latency under the staging's HBM loads
  // (one memory round trip); slots from nvalid on hold no token yet and are
  // staged as zero rows ----
  static_assert(D <= 256 && DV <= 256, "one element of a token row per thread");
  KeyBankRows<T, D> kb;
  if constexpr (PRE) kb.load(om, M, tid);
  RingStage<T, W, D, false> rgr;
  RingStage<T, W, DV, true> rgu;
  rgr.load(rr, rt, slot, w, tid);
  rgu.load(ru, ut, slot, w, tid);
  // (r_t and u_t are kept for the ring slot written at the end)
  const T xq = qt[min(tid, D - 1)], xk = kt[min(tid, D - 1)], xv = vt[min(tid, DV - 1)];
  const T xr = rt[min(tid, D - 1)], xu = ut[min(tid, DV - 1)];
  const float Rold = A.rho[sh];
  if (tid < D) {
    sq[tid] = tof(xq);
    sk[tid] = tof(xk);
  }
  if (tid < DV) sv[tid] = tof(xv);
  rgr.store(sRr, D + PAD, nvalid, tid);
  rgu.store(sUt, W + PAD, nvalid, tid);
  if constexpr (!PRE) stage_omega<T, D, M>(sOm, om, tid);
  // the state rows this thread updates, issued once the staging has been
  // waited for: the memory counter drains in issue order, so no wait before
  // the update includes them, and they arrive under the GEMV, the logits and
  // the exponentials
  if constexpr (PRE) {
    if (wv < PT) {
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt)
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) mreg[dt][vv] = Ms[(size_t)(wv * 32 + crow(vv, h)) * DV + dt * 32 + col];
    }
  }
  __syncthreads();

  // ---- key features of k_t (float32 GEMV) and the frame update; with one
  // feature tile per wave the Omega rows of the GEMV also give the logits'
  // operand fragments (no LDS copy of the bank) ----
  typename F::frag omf[PRE ? D / F::KS : 1];
  float rho_t;
  if constexpr (PRE) rho_t = key_log2_features_rows<T, D, M, PRE>(kb, sk, schi, sred, omf);
  else rho_t = key_log2_features<T, D, M, PRE>(sk, om, schi, sred, omf);
  const float lam = tid < M ? schi[tid] : kNegInf;   // each thread rewrites only its own entry below
  const float Rn = fmaxf(Rold, rho_t);
  const float sa = fast_exp2(Rold - Rn);          // 0 for an empty state (R = -inf)
  if (tid < M) {
    float chi = fast_exp2(lam - Rn) * rsqrtf((float)M);
    schi[tid] = chi;
    float an = sa * a_old + chi;
    san[tid] = an;
    as[tid] = an;
  }
  // ---- composite-query logits, lanes <-> feature p, registers <-> anchor ----
  f32x16 acc[PTW][NA];
  float nz[NA];
#pragma unroll
  for (int pi = 0; pi < PTW; ++pi)
#pragma unroll
    for (int ct = 0; ct < NA; ++ct) acc[pi][ct] = zero16();
#pragma unroll
  for (int ct = 0; ct < NA; ++ct) nz[ct] = 0.0f;
  // (anchors past nvalid read zero ring rows, so z = 0 there without a mask)
#pragma unroll
  for (int ct = 0; ct < NA; ++ct) {
    const int c = ct * 32 + col;
    const bool valid = c < nvalid;
#pragma unroll
    for (int ks = 0; ks < D / F::KS; ++ks) {
      no_hoist();                                 // the step's q reads stay in the step
      const int k0 = ks * F::KS + h * F::KPL;
      typename F::frag rf = F::ld(sRr + c * (D + PAD), k0), zf;
      composite_query<T>(sq + k0, rf, nz[ct], zf);
      if constexpr (PRE) {
        if (wv < PT) acc[0][ct] = F::mma(zf, omf[ks], acc[0][ct]);
      } else {
#pragma unroll
        for (int pi = 0; pi < PTW; ++pi) {
          const int pt = wv + 4 * pi;
          if (pt < PT)
            acc[pi][ct] = F::mma(zf, F::ld(sOm + (pt * 32 + col) * (D + PAD), k0), acc[pi][ct]);
        }
      }
    }
    nz[ct] = half_swap_add(nz[ct]);
    if (wv == 0 && h == 0) snz[c] = valid ? -0.5f * kLog2e * nz[ct] : kNegInf;
  }
  __syncthreads();
  // row maximum over valid (anchor, feature)
  float tm = kNegInf;
#pragma unroll
  for (int pi = 0; pi < PTW; ++pi) {
    if (wv + 4 * pi >= PT) continue;
#pragma unroll
    for (int ct = 0; ct < NA; ++ct)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = acc[pi][ct][v] + snz[ct * 32 + crow(v, h)];
        acc[pi][ct][v] = x;
        tm = fmaxf(tm, x);
      }
  }
  tm = wave_max(tm);
  if (l == 0) sred[8 + wv] = tm;
  __syncthreads();
  const float L = fmaxf(fmaxf(sred[8], sred[9]), fmaxf(sred[10], sred[11]));
  // psi, Z, then W = Psi^T U and N = sum_p M'[p,:] (*) W[p,:] with the state update
  float zpart = 0.0f;
  float npart[DV / 32];
#pragma unroll
  for (int dt = 0; dt < DV / 32; ++dt) npart[dt] = 0.0f;
#pragma unroll
  for (int pi = 0; pi < PTW; ++pi) {
    const int pt = wv + 4 * pi;
    if (pt >= PT) continue;
    const float anp = san[pt * 32 + col];
#pragma unroll
    for (int ct = 0; ct < NA; ++ct)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float psi = fast_exp2(acc[pi][ct][v] - L);
        acc[pi][ct][v] = psi;
        zpart += psi * anp;
      }
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) {
      no_hoist();
      f32x16 accW = zero16();
      const T* urow = sUt + (dt * 32 + col) * (W + PAD);
#pragma unroll
      for (int ct = 0; ct < NA; ++ct)
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp)
          accW = F::mma(F::cfrag(acc[pi][ct], sp), F::ldc(urow, ct * 32, sp, h), accW);
      // accW: lanes <-> d, registers <-> p
      const int d = dt * 32 + col;
      const float vd = sv[d];
      float np = 0.0f;
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) {
        const int p = pt * 32 + crow(vv, h);
        float* mp = Ms + (size_t)p * DV + d;
        float mold;
        if constexpr (PRE) mold = mreg[dt][vv];
        else mold = *mp;
        float mnew = sa * mold + schi[p] * vd;
        *mp = mnew;
        np += mnew * accW[vv];
      }
      npart[dt] += np;
    }
  }
  // (feature tile pt belongs to wave pt mod 4, so every state row is updated once)
  zpart = wave_sum(zpart);
  if (l == 0) sred[16 + wv] = zpart;
#pragma unroll
  for (int dt = 0; dt < DV / 32; ++dt) {
    float nn = half_swap_add(npart[dt]);
    if (h == 0) sN[wv * DV + dt * 32 + col] = nn;
  }
  __syncthreads();
  const float Z = (sred[16] + sred[17]) + (sred[18] + sred[19]);
  const float inv = 1.0f / (Z + A.eps);
  for (int d = tid; d < DV; d += 256) {
    float N = (sN[d] + sN[DV + d]) + (sN[2 * DV + d] + sN[3 * DV + d]);
    ((T*)A.out)[(size_t)sh * DV + d] = (T)(N * inv);
  }
  // ring slot and frame
  if (tid < D) rr[(size_t)slot * D + tid] = xr;
  if (tid < DV) ru[(size_t)slot * DV + tid] = xu;
  if (tid == 0) A.rho[sh] = Rn;
}

// ---------------------------------------------------------------------------
// Chunked decode: NT tokens per sequence in one launch (token j of sequence s
// is position pos[s] + j).  The same per-token step as k_decode, but the
// state stays on chip for the whole chunk: the ring anchors live in LDS and
// are overwritten slot by slot, a lives in the registers of the threads that
// own a feature, and M (for m <= 128) lives in the registers of the threads
// that update it, so each state element is read and written once per chunk
// instead of once per token.  For m = 256 M is streamed through global memory
// per token as in k_decode.
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M, int NA>
__global__ __launch_bounds__(256) void k_decode_chunk(DecArgs A, int NTOK) {
  using F = MF<T>;
  using C = DCfg<T, D, DV, M, NA>;
  constexpr int PAD = C::PAD, W = C::W;
  constexpr int PT = M / 32;                  // feature tiles
  constexpr int PTW = (PT + 3) / 4;           // feature tiles per wave
  constexpr bool RES = PTW == 1;              // M held in registers across the chunk
  static_assert(C::BYTES <= 160 * 1024, "decode LDS budget");
  __shared__ __align__(16) char smem[C::BYTES];
  T* sOm = (T*)(smem + C::oOm);
  T* sRr = (T*)(smem + C::oRr);
  T* sUt = (T*)(smem + C::oUt);
  float* sq = (float*)(smem + C::oQ);
  float* sk = (float*)(smem + C::oK);
  float* sv = (float*)(smem + C::oV);
  float* schi = (float*)(smem + C::oChi);
  float* san = (float*)(smem + C::oAn);
  float* snz = (float*)(smem + C::oNz);
  float* sred = (float*)(smem + C::oRed);
  float* sN = (float*)(smem + C::oN);

  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  const int sh = blockIdx.x, H = A.H, w = A.w;
  const int s = sh / H, hh = sh % H;
  const int64_t t0 = A.pos[s];
  T* rr = (T*)A.ring_r + (size_t)sh * w * D;
  T* ru = (T*)A.ring_u + (size_t)sh * w * DV;
  const float* om = A.omega + (size_t)hh * M * D;
  float* Ms = A.M + (size_t)sh * M * DV;
  float* as = A.a + (size_t)sh * M;

  // ring, Omega and the state, once per chunk; while t0 < w the slots t0 .. w-1
  // hold no token yet: they are staged as zero rows and the chunk's tokens
  // fill them in order
  const int nv0 = (int)(t0 < w ? t0 : w);
  {
    RingStage<T, W, D, false> rgr;
    RingStage<T, W, DV, true> rgu;
    rgr.load(rr, nullptr, 0, w, tid);
    rgu.load(ru, nullptr, 0, w, tid);
    rgr.store(sRr, D + PAD, nv0, tid);
    rgu.store(sUt, W + PAD, nv0, tid);
  }
  stage_omega<T, D, M>(sOm, om, tid);
  float areg = (tid < M) ? as[tid] : 0.0f;
  float R = A.rho[sh];
  float Mreg[RES ? DV / 32 : 1][16];
  if constexpr (RES) {
    if (wv < PT) {
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt)
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) Mreg[dt][vv] = Ms[(size_t)(wv * 32 + crow(vv, h)) * DV + dt * 32 + col];
    }
  }

  // a token's q, k, r (element tid of D) and v, u (element tid of DV) are
  // loaded one token ahead into registers: their latency then overlaps the
  // previous token's work instead of opening each token's chain.  Every
  // thread loads (index clamped into the row), so no load sits under a branch.
  static_assert(D <= 256 && DV <= 256, "one element of a token row per thread");
  const int iD = min(tid, D - 1), iV = min(tid, DV - 1);
  T xq, xk, xr, xv, xu;
  auto fetch_token = [&](int j) {
    const size_t tok = (size_t)sh * NTOK + j;
    xq = ((const T*)A.q)[tok * D + iD];
    xk = ((const T*)A.k)[tok * D + iD];
    xr = ((const T*)A.r)[tok * D + iD];
    xv = ((const T*)A.v)[tok * DV + iV];
    xu = ((const T*)A.u)[tok * DV + iV];
  };
  fetch_token(0);

#pragma unroll 1
  for (int j = 0; j < NTOK; ++j) {
    const int64_t t = t0 + j;
    const int slot = (int)(t % w);
    const int nvalid = (int)((t + 1 < w) ? t + 1 : w);
    const size_t tok = (size_t)sh * NTOK + j;
    __syncthreads();                              // the previous token is done with LDS
    if (tid < D) {
      sq[tid] = tof(xq);
      sk[tid] = tof(xk);
      sRr[slot * (D + PAD) + tid] = xr;
    }
    if (tid < DV) {
      sv[tid] = tof(xv);
      sUt[tid * (W + PAD) + F::sigma(slot)] = xu;
    }
    __syncthreads();

    // key features of k_t and the frame update
    const float rho_t = key_log2_features<T, D, M, false>(sk, om, schi, sred, nullptr);
    // the next token's rows, issued after the bank loads of the key GEMV (the
    // memory counter drains in issue order: issued before them, they would be
    // waited for with them)
    if (j + 1 < NTOK) fetch_token(j + 1);
    const float lam = tid < M ? schi[tid] : kNegInf;
    const float Rn = fmaxf(R, rho_t);
    const float sa = fast_exp2(R - Rn);
    if (tid < M) {
      const float chi = fast_exp2(lam - Rn) * rsqrtf((float)M);
      schi[tid] = chi;
      areg = sa * areg + chi;
      san[tid] = areg;
    }
    // composite-query logits (lanes <-> feature, registers <-> anchor)
    f32x16 acc[PTW][NA];
    float nz[NA];
#pragma unroll
    for (int pi = 0; pi < PTW; ++pi)
#pragma unroll
      for (int ct = 0; ct < NA; ++ct) acc[pi][ct] = zero16();
#pragma unroll
    for (int ct = 0; ct < NA; ++ct) nz[ct] = 0.0f;
#pragma unroll
    for (int ct = 0; ct < NA; ++ct) {
      const int c = ct * 32 + col;
      const bool valid = c < nvalid;
#pragma unroll 2
      for (int ks = 0; ks < D / F::KS; ++ks) {
        no_hoist();
        const int k0 = ks * F::KS + h * F::KPL;
        typename F::frag rf = F::ld(sRr + c * (D + PAD), k0), zf;
        composite_query<T>(sq + k0, rf, nz[ct], zf);
#pragma unroll
        for (int pi = 0; pi < PTW; ++pi) {
          const int pt = wv + 4 * pi;
          if (pt < PT)
            acc[pi][ct] = F::mma(zf, F::ld(sOm + (pt * 32 + col) * (D + PAD), k0), acc[pi][ct]);
        }
      }
      nz[ct] = half_swap_add(nz[ct]);
      if (wv == 0 && h == 0) snz[c] = valid ? -0.5f * kLog2e * nz[ct] : kNegInf;
    }
    __syncthreads();
    float tm = kNegInf;
#pragma unroll
    for (int pi = 0; pi < PTW; ++pi) {
      if (wv + 4 * pi >= PT) continue;
#pragma unroll
      for (int ct = 0; ct < NA; ++ct)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float x = acc[pi][ct][v] + snz[ct * 32 + crow(v, h)];
          acc[pi][ct][v] = x;
          tm = fmaxf(tm, x);
        }
    }
    tm = wave_max(tm);
    if (l == 0) sred[8 + wv] = tm;
    __syncthreads();
    const float L = fmaxf(fmaxf(sred[8], sred[9]), fmaxf(sred[10], sred[11]));
    float zpart = 0.0f;
    float npart[DV / 32];
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) npart[dt] = 0.0f;
#pragma unroll
    for (int pi = 0; pi < PTW; ++pi) {
      const int pt = wv + 4 * pi;
      if (pt >= PT) continue;
      const float anp = san[pt * 32 + col];
#pragma unroll
      for (int ct = 0; ct < NA; ++ct)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float psi = fast_exp2(acc[pi][ct][v] - L);
          acc[pi][ct][v] = psi;
          zpart += psi * anp;
        }
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt) {
        f32x16 accW = zero16();
        const T* urow = sUt + (dt * 32 + col) * (W + PAD);
#pragma unroll
        for (int ct = 0; ct < NA; ++ct)
#pragma unroll
          for (int sp = 0; sp < F::CSTEPS; ++sp)
            accW = F::mma(F::cfrag(acc[pi][ct], sp), F::ldc(urow, ct * 32, sp, h), accW);
        const int d = dt * 32 + col;
        const float vd = sv[d];
        float np = 0.0f;
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) {
          const int p = pt * 32 + crow(vv, h);
          float mnew;
          if constexpr (RES) {
            mnew = sa * Mreg[dt][vv] + schi[p] * vd;
            Mreg[dt][vv] = mnew;
          } else {
            float* mp = Ms + (size_t)p * DV + d;
            mnew = sa * (*mp) + schi[p] * vd;
            *mp = mnew;
          }
          np += mnew * accW[vv];
        }
        npart[dt] += np;
      }
    }
    zpart = wave_sum(zpart);
    if (l == 0) sred[16 + wv] = zpart;
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) {
      const float nn = half_swap_add(npart[dt]);
      if (h == 0) sN[wv * DV + dt * 32 + col] = nn;
    }
    __syncthreads();
    const float Z = (sred[16] + sred[17]) + (sred[18] + sred[19]);
    const float inv = 1.0f / (Z + A.eps);
    for (int d = tid; d < DV; d += 256) {
      const float N = (sN[d] + sN[DV + d]) + (sN[2 * DV + d] + sN[3 * DV + d]);
      ((T*)A.out)[tok * DV + d] = (T)(N * inv);
    }
    R = Rn;
  }

  // state and ring back to global memory
  if constexpr (RES) {
    if (wv < PT) {
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt)
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) Ms[(size_t)(wv * 32 + crow(vv, h)) * DV + dt * 32 + col] = Mreg[dt][vv];
    }
  }
  if (tid < M) as[tid] = areg;
  if (tid == 0) A.rho[sh] = R;
  // the last min(NTOK, w) tokens stay in the ring: their rows are read from the
  // LDS ring (written by their tokens and made visible by the tokens' barriers),
  // not again from global memory (a global load per row, each waited for)
  const int jlo = NTOK > w ? NTOK - w : 0;
  for (int j = jlo; j < NTOK; ++j) {
    const int slot = (int)((t0 + j) % w);
    for (int e = tid; e < D; e += 256) rr[(size_t)slot * D + e] = sRr[slot * (D + PAD) + e];
    for (int e = tid; e < DV; e += 256) ru[(size_t)slot * DV + e] = sUt[e * (W + PAD) + F::sigma(slot)];
  }
}

// pos[s] += step after every head of sequence s has read it
__global__ __launch_bounds__(256) void k_decode_advance(int64_t* pos, int64_t S, int step) {
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < S) pos[i] += step;
}

template <typename T, int D, int DV, int M, int NA>
static int run_decode(int64_t S, DecArgs a, int ntok, hipStream_t st) {
  // the caller bounds S*H by kMaxDecodeGroups (one workgroup each)
  (void)hipGetLastError();                             // an earlier call's error is not this one's
  if (ntok == 1) {
    ProfScope ps("decode", st);
    k_decode<T, D, DV, M, NA><<<(unsigned)(S * a.H), 256, 0, st>>>(a);
  } else {
    ProfScope ps("decode_chunk", st);
    k_decode_chunk<T, D, DV, M, NA><<<(unsigned)(S * a.H), 256, 0, st>>>(a, ntok);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {                               // pos must not advance past a step not taken
    set_error("decode launch failed: %s", hipGetErrorString(e));
    return -4;
  }
  k_decode_advance<<<(unsigned)((S + 255) / 256), 256, 0, st>>>(a.pos, S, ntok);
  e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("decode position update launch failed: %s", hipGetErrorString(e));
    return -4;
  }
  return 0;
}

#define LS_DEC_CASES(X)   \
  X(bf16, 32, 32, 32)     \
  X(bf16, 64, 64, 64)     \
  X(bf16, 64, 64, 128)    \
  X(bf16, 128, 128, 64)   \
  X(bf16, 128, 128, 128)  \
  X(bf16, 128, 128, 256)  \
  X(float, 32, 32, 32)    \
  X(float, 32, 32, 64)    \
  X(float, 64, 64, 32)    \
  X(float, 64, 64, 64)

int launch_decode(int64_t S, int H, int ntok, int D, int Dv, int m, int w, int dtype, float eps,
                  const void* q, const void* k, const void* v, const void* r, const void* u,
                  const float* omega, float* M, float* a, float* rho, void* ring_r, void* ring_u,
                  int64_t* pos, void* out, hipStream_t st) {
  DecArgs A;
  A.q = q; A.k = k; A.v = v; A.r = r; A.u = u; A.omega = omega;
  A.M = M; A.a = a; A.rho = rho; A.ring_r = ring_r; A.ring_u = ring_u; A.pos = pos; A.out = out;
  A.H = H; A.w = w; A.eps = eps;
  const int NA = (w + 31) / 32;
#define X(T, D_, DV_, M_)                                                              \
  if (dtype == (sizeof(T) == 2 ? 1 : 0) && D == D_ && Dv == DV_ && m == M_) {          \
    if (NA == 1) return run_decode<T, D_, DV_, M_, 1>(S, A, ntok, st);                 \
    if (NA == 2) return run_decode<T, D_, DV_, M_, 2>(S, A, ntok, st);                 \
    if constexpr (wide_window_ok(sizeof(T) == 2 ? 1 : 0, D_, M_, 3)) {                  \
      if (NA == 3) return run_decode<T, D_, DV_, M_, 3>(S, A, ntok, st);               \
    }                                                                                  \
    if constexpr (wide_window_ok(sizeof(T) == 2 ? 1 : 0, D_, M_, 4)) {                  \
      if (NA == 4) return run_decode<T, D_, DV_, M_, 4>(S, A, ntok, st);               \
    }                                                                                  \
  }
  LS_DEC_CASES(X)
#undef X
  set_error("decode: unsupported shape (dtype=%d D=%d Dv=%d m=%d)", dtype, D, Dv, m);
  return -2;
}

}  // namespace linsimp
