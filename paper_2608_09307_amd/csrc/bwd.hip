// LinSimp backward on gfx950: exact gradient of sum_i dO_i . out_i with the
// stabilising shifts held constant (they cancel in the ratio, App. B.2).
//
// Per row i (log2 frames as in the forward; psi = 2^(ell - L_i), the query
// feature without 1/sqrt(m); M^(i), a^(i) the state of row i in frame R_i):
//   dN = g / (Z + eps),  dZ = -(g . out) / (Z + eps)
//   per anchor c:  dA_c = dN (*) u_c,  du_c += dN (*) A_c,  A_c = psi_c^T M^(i)
//                  dpsi_c = M^(i) dA_c + dZ a^(i)
//                  dell_c = dpsi_c (*) psi_c            (natural-log derivative)
//                  dz_c = Omega^T dell_c - (sum_p dell_cp) z_c    (d ell/d z = omega - z, App. C)
//                  dq_i += dz_c (*) r_c,  dr_c += dz_c (*) q_i
//   state:         dM^(i) = sum_c psi_c dA_c^T,  da^(i) = dZ sum_c psi_c
// M^(i) = sb_i M_b + sum_{j in chunk, j<=i} 2^(R_j-R_i) chi_j v_j^T, so the state
// gradient splits into the chunk boundary (GB_b = sum_i sb_i dM^(i), carried to
// earlier chunks by a reverse scan: App. C "Backward state sweep") and the
// intra-chunk tail (dchi_j, dv_j from rows j <= i of the same chunk).  The key
// feature map is then differentiated: dlambda = dchi (*) chi,
// dk = Omega^T dlambda - (sum_p dlambda_p) k.
//
// Kernels:
//   k_bwd_rowprep  row scalars 1/(Z+eps) and dZ
//   k_bwd_du       anchor sweep 1: du
//   k_bwd_dqdr     anchor sweep 2: dr (anchor side) and per-tile partials of dq
//   k_bwd_state    state sweep: GB_b, gb_b and the intra-chunk dchi, dv
//   k_bwd_revscan  reverse exclusive scan of (GB, gb) with the frame monoid
//   k_bwd_keys     key side: dk, dv
//   k_bwd_final*   float32 partials -> output dtype
// The anchor sweeps are anchor-stationary: a workgroup owns 32 anchors and
// walks the rows that see them, so du and dr are summed in registers (no
// atomics anywhere); dq of a row is the sum of its anchor tiles' partials.
#include <type_traits>

#include "common.h"
#include "linsimp_internal.h"
#include "prof.h"

namespace linsimp {


struct BwdArgs {
  const void *q, *k, *v, *r, *u;
  const float* omega;
  const void* out;
  const float* stats;
  const void* dout;
  void *dq, *dk, *dv, *dr, *du;
  const void* omq;
  const void* omk;
  const void* omh;
  const float* states;
  const void* states16;
  const float* rex;
  float* gst;       // [BH][nch][M*DV + M]  GB_b, then Ghat_b
  float* dchi;      // [BH][n][M]           intra-chunk key-feature gradient
  float* dvin;      // [NFB][BH][n][DV]     intra-chunk value gradient
  float* du32;      // [NFB][BH][n][DV]     per feature block (NFB > 1)
  float* dr32;      // [NFB][BH][n][D]      per feature block (NFB > 1)
  float* dq32;      // [NFB][NS][BH][n][D]  per anchor tile (slot = row chunk - tile)
  void* chi;        // [BH][n][M]           key features, p permuted in 16-blocks
  float* rj;        // [BH][n]              running key frame R_j
  float* rowstat;   // [BH][n][2]: 1/(Z+eps), dZ
  int H, n, w, nch, BH;
  float eps;
};

static constexpr float kLn2 = 0.6931471805599453f;


// ---------------------------------------------------------------------------
// prep: row scalars and zeroed float32 accumulators
// ---------------------------------------------------------------------------
// One row per LPR lanes, each lane one 16-byte piece of dO and of out.
template <typename T, int DV>
__global__ __launch_bounds__(256) void k_bwd_rowprep(BwdArgs a) {
  constexpr int VE = 16 / sizeof(T);
  constexpr int LPR = DV / VE;                 // lanes per row (a power of two, <= 32)
  typedef T V __attribute__((ext_vector_type(VE)));
  const size_t rows = (size_t)a.BH * a.n;
  const size_t row = (size_t)blockIdx.x * (256 / LPR) + threadIdx.x / LPR;
  const int lane = threadIdx.x % LPR;
  const bool act = row < rows;
  const size_t rr = act ? row : rows - 1;
  const V g = *(const V*)((const T*)a.dout + rr * DV + lane * VE);
  const V o = *(const V*)((const T*)a.out + rr * DV + lane * VE);
  float s = 0.0f;
#pragma unroll
  for (int e = 0; e < VE; ++e) s += tof(g[e]) * tof(o[e]);
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, LPR);
  if (act && lane == 0) {
    const float inv = 1.0f / (a.stats[row * 2 + 1] + a.eps);
    a.rowstat[row * 2 + 0] = inv;
    a.rowstat[row * 2 + 1] = -s * inv;
  }
}


// ---------------------------------------------------------------------------
// Anchor-stationary sweeps.  A workgroup owns the 32 anchors [c0, c0 + 32) of
// one sequence and one feature block, and walks the row chunks that can see
// them (rows c0 .. c0 + 31 + w - 1); in the dq/dr sweep each wave takes
// every eighth row of a chunk (du, below, stages the three chunks at once and
// pairs rows).  Per (row, anchor tile) the query features psi[p, c] are formed with
// lanes <-> anchor (registers <-> feature), exactly as in the forward readout,
// and the anchor-side sums stay in registers; the waves' sums are added once
// at the end.
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M, int NA>
struct AsCfg {
  static constexpr int PAD = MF<T>::PAD;
  static constexpr int FB = M < 128 ? M : 128;
  static constexpr int NFB = M / FB;
  static constexpr int NW = 8;
  static constexpr int ES = sizeof(T);
  static constexpr int a16(int x) { return (x + 15) & ~15; }
  static constexpr int mx(int x, int y) { return x > y ? x : y; }
  static constexpr int oOm = 0;                                             // Omega block [p][D]
  static constexpr int oM = oOm + a16(FB * (D + PAD) * ES);                 // boundary M ([d][sigma(p)] or [p][d])
  static constexpr int TPF = tr_pad<T, FB>(), TPD = tr_pad<T, D>();
  // row pitches: chi and r are read transposed
  static constexpr int CST = FB + TPF;
  static constexpr int VST = DV + PAD;
  static constexpr int RST = D + TPD;
  static constexpr int oChi = oM + a16(mx(DV * (FB + PAD), FB * (DV + PAD)) * ES);   // chi [j][sigma(p)]
  static constexpr int oV = oChi + a16(32 * CST * ES);                      // V [j][d]
  static constexpr int oQ = oV + a16(32 * VST * ES);                        // q rows of the chunk
  static constexpr int oR = oQ + a16(32 * (D + PAD) * ES);                  // r of the anchor tile
  static constexpr int oU = oR + a16(32 * RST * ES);                        // u of the anchor tile
  static constexpr int oRj = oU + a16(32 * (DV + PAD) * ES);                // R_j of the chunk
  static constexpr int oRat = oRj + a16(32 * 4);                            // 2^(R_j - Rref) of the chunk
  static constexpr int oA = oRat + a16(32 * 4);                             // boundary a
  static constexpr int oW = oA + a16(FB * 4);                               // per wave: dN (DV), s_c (32)
  static constexpr int oOb = oW + a16(NW * (DV + 32) * 4);                 // Omega*log2 e, operand type (dz)
  static constexpr int BYTES0 = oOb + a16(FB * (D + TPD) * ES);
  static constexpr int RED = (NW / 2) * 32 * mx(DV, D) * 4;                 // end-of-sweep reduction
  static constexpr int BYTES = mx(BYTES0, RED);
};

// Sum the waves' 32 x (32 NT) accumulators into wave 0 through LDS (the
// caller has finished with the other shared buffers).
template <int NT>
LS_DEV void reduce_waves(f32x16 (&acc)[NT], float* red, int wv, int NW) {
  const int l = lane_id(), col = l & 31, h = l >> 5;
  constexpr int W = 32 * NT;
  for (int half = NW / 2; half >= 1; half >>= 1) {
    __syncthreads();
    if (wv >= half && wv < 2 * half) {
      float* dst = red + (size_t)(wv - half) * 32 * W;
#pragma unroll
      for (int dt = 0; dt < NT; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) dst[crow(v, h) * W + dt * 32 + col] = acc[dt][v];
    }
    __syncthreads();
    if (wv < half) {
      const float* src = red + (size_t)wv * 32 * W;
#pragma unroll
      for (int dt = 0; dt < NT; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[dt][v] += src[crow(v, h) * W + dt * 32 + col];
    }
  }
}

// psi[p, c] of one (row, anchor tile) pair: log2 features of z = q_i (*) r_c
// against the block's Omega rows, shifted by L_i, masked anchors give 0.
// Psi fragments are operand fragments (MF<T>::frag) where psi feeds the
// matrix cores, or f16x8 where it only scales (psi <= 1 after the shift).
LS_DEV void to_frag(bf16x8& f, const f32x16& acc, int sp) { f = MF<bf16>::cfrag(acc, sp); }
LS_DEV void to_frag(float& f, const f32x16& acc, int sp) { f = MF<float>::cfrag(acc, sp); }
LS_DEV void to_frag(f16x8& f, const f32x16& acc, int sp) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const f16x2 x = __builtin_bit_cast(f16x2, __builtin_amdgcn_cvt_pkrtz(acc[8 * sp + 2 * e], acc[8 * sp + 2 * e + 1]));
    f[2 * e] = x[0];
    f[2 * e + 1] = x[1];
  }
}

template <typename T, int D, int FB, typename PF = typename MF<T>::frag>
LS_DEV void query_features(PF (&pf)[FB / 32][MF<T>::CSTEPS], const T* qrow,
                           const T* rrow, const T* sOm, bool valid, float Li) {
  using F = MF<T>;
  constexpr int PAD = F::PAD;
  const int l = lane_id(), col = l & 31, h = l >> 5;
  f32x16 accL[FB / 32];
  float nz;
  if constexpr (sizeof(T) == 2) {
    // bf16 inputs: q, r and Omega*log2(e) sit in LDS as f16 (see logits_f16)
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
  // masked anchors: z is finite (zero-filled rows) and the offset removes them
  const float off = valid ? -0.5f * kLog2e * nz - Li : kNegInf;
#pragma unroll
  for (int pt = 0; pt < FB / 32; ++pt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) accL[pt][v] = fast_exp2(accL[pt][v] + off);
#pragma unroll
    for (int sp = 0; sp < F::CSTEPS; ++sp) to_frag(pf[pt][sp], accL[pt], sp);
  }
}

// frame ratios 2^(R_j - Rref) of the chunk's rows (sRat), masked to j <= t, for
// the registers' rows j (all sixteen read, later rows then zeroed: no branches)
LS_DEV void masked_ratios(float (&sj)[16], const float* sRat, int t) {
  const int h = lane_id() >> 5;
  const float* sh = sRat + 4 * h;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const f32x4 r4 = *(const f32x4*)(sh + 8 * g);
#pragma unroll
    for (int e = 0; e < 4; ++e) sj[4 * g + e] = (8 * g + 4 * h + e <= t) ? r4[e] : 0.0f;
  }
}

// ---------------------------------------------------------------------------
// k_bwd_du: du_c = sum_i dN_i (*) A_ic,  A_ic = psi_ic^T M^(i)  (regs <-> anchor,
// lanes <-> d).  A workgroup stages once the boundary state M_b of its own
// chunk kt and the key features, values and queries of chunks kt .. kt+NA
// (NA = ceil(w / 32) anchor tiles per row); the state of any row i that sees
// the tile is then the boundary part plus a tail of at most NA + 1 chunks,
//   M^(i) = 2^(Rex_kt - R_i) M_b + sum_{c0 <= j <= i} 2^(R_j - R_i) chi_j v_j^T
// (computed in the reference frame Rref = Rex_kt, the row factor 2^(Rref - R_i)
// applied to dN_i once).
// Row t of chunk kt sees anchors c <= t of the tile and row t of chunk kt+NA
// anchors c > t only (w <= 32 NA): the two run as one pair, each lane c taking
// the row that sees anchor c, so the logits, features and boundary product are
// formed once for both.  Rows of chunks kt+1 .. kt+NA-1 run one at a time.
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M, int NA>
struct DuCfg {
  static constexpr int PAD = MF<T>::PAD;
  static constexpr int FB = M < 128 ? M : 128;
  static constexpr int NW = 8;
  static constexpr int NCH = NA + 1;                         // staged row chunks
  static constexpr int ROWS = 32 * NCH;
  static constexpr int ES = sizeof(T);
  static constexpr int a16(int x) { return (x + 15) & ~15; }
  static constexpr int mx(int x, int y) { return x > y ? x : y; }
  static constexpr int CST = FB + PAD;                       // chi [j][sigma(p)]
  static constexpr int VST = DV + tr_pad<T, DV>();           // V [j][d] (read transposed)
  static constexpr int oOm = 0;                              // Omega block [p][D]
  static constexpr int oM = oOm + a16(FB * (D + PAD) * ES);  // M_b^T [d][sigma(p)]
  static constexpr int oChi = oM + a16(DV * (FB + PAD) * ES);
  static constexpr int oV = oChi + a16(ROWS * CST * ES);
  static constexpr int oQ = oV + a16(ROWS * VST * ES);
  static constexpr int oR = oQ + a16(ROWS * (D + PAD) * ES); // r of the anchor tile
  static constexpr int oRj = oR + a16(32 * (D + PAD) * ES);  // R_j of the staged rows
  static constexpr int oRat = oRj + a16(ROWS * 4);           // 2^(R_j - Rref) of the staged rows
  static constexpr int BYTES0 = oRat + a16(ROWS * 4);
  static constexpr int RED = (NW / 2) * 32 * DV * 4;         // end-of-sweep reduction
  static constexpr int BYTES = mx(BYTES0, RED);
};

template <typename T, int D, int DV, int M, int NA>
__global__ __launch_bounds__(64 * 8) void k_bwd_du(BwdArgs a) {
  using F = MF<T>;
  using C = DuCfg<T, D, DV, M, NA>;
  constexpr int PAD = C::PAD, FB = C::FB, NW = C::NW, CST = C::CST, VST = C::VST, ROWS = C::ROWS;
  constexpr int NT = 64 * NW;
  constexpr int S = M * DV + M;
  static_assert(C::BYTES <= 160 * 1024, "du LDS budget");
  __shared__ __align__(16) char smem[C::BYTES];
  T* sOm = (T*)(smem + C::oOm);
  T* sMt = (T*)(smem + C::oM);
  T* sChi = (T*)(smem + C::oChi);
  T* sV = (T*)(smem + C::oV);
  T* sQ = (T*)(smem + C::oQ);
  T* sR = (T*)(smem + C::oR);
  float* sRj = (float*)(smem + C::oRj);
  float* sRat = (float*)(smem + C::oRat);

  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  const int2 gxy = xcd_grid_xy();
  const int kt = gxy.x, bh = gxy.y, hh = bh % a.H, n = a.n, nch = a.nch, fb = blockIdx.z;
  const int c0 = kt * 32, w = a.w;
  const size_t seq = (size_t)bh * n;
  const T* qs = (const T*)a.q + seq * D;
  const T* vs = (const T*)a.v + seq * DV;
  const T* rs_ = (const T*)a.r + seq * D;
  const T* gs = (const T*)a.dout + seq * DV;
  const T* chis = (const T*)a.chi + seq * M + fb * FB;
  const T* omq_h = (const T*)a.omq + (size_t)hh * M * D;
  const bool has_bnd = kt > 0;
  const float Rexb = a.rex[(size_t)bh * (nch + 1) + kt];
  // reference frame of the staged rows: the boundary frame (the first chunk,
  // whose boundary state is zero, takes R of its first row); then
  //   A_ic = 2^(Rref - R_i) [psi_c^T M_b + sum_{c0 <= j <= i} 2^(R_j - Rref) (chi_j . psi_c) v_j^T]
  // and the row factor 2^(Rref - R_i) goes into dN_i
  const float Rref = uniform(has_bnd ? Rexb : a.rj[seq + c0]);

  // ---- staging, once per workgroup ----
  {
    // Omega block, r of the tile and the boundary state (zero for the first chunk)
    StageState<FB, DV, NT, true> sm;
    StageRowsT<T, FB, DV, NT> sm16;
    if constexpr (sizeof(T) == 2) {
      if (has_bnd) sm16.load((const T*)a.states16 + (((size_t)bh * nch + kt) * M + (size_t)fb * FB) * DV, DV, 0, 0, FB, tid);
    } else {
      if (has_bnd) sm.load(a.states + ((size_t)bh * nch + kt) * S + (size_t)fb * FB * DV, tid);
    }
    if constexpr (sizeof(T) == 2) {
      StageRows<f16, FB, D, NT> so;
      StageRows<T, 32, D, NT> sr;
      so.load((const f16*)a.omh + ((size_t)hh * M + (size_t)fb * FB) * D, D, 0, 0, FB, tid);
      sr.load(rs_, D, c0, 0, n, tid);
      so.store((f16*)sOm, D + PAD, 0, 0, FB, tid);
      sr.store((f16*)sR, D + PAD, c0, 0, n, tid);
      sm16.store(0, 0, FB, tid, [&](int p, int d0, const typename StageRowsT<T, FB, DV, NT>::V4& x) {
#pragma unroll
        for (int e = 0; e < 4; ++e) sMt[(d0 + e) * (FB + PAD) + F::sigma(p)] = has_bnd ? x[e] : (T)0.0f;
      });
    } else {
      StageRows<T, FB, D, NT> so;
      StageRows<T, 32, D, NT> sr;
      so.load(omq_h + (size_t)fb * FB * D, D, 0, 0, FB, tid);
      sr.load(rs_, D, c0, 0, n, tid);
      so.store(sOm, D + PAD, 0, 0, FB, tid);
      sr.store(sR, D + PAD, c0, 0, n, tid);
      sm.store(tid, [&](int p, int d0, const f32x4& x) {
#pragma unroll
        for (int e = 0; e < 4; ++e) sMt[(d0 + e) * (FB + PAD) + F::sigma(p)] = has_bnd ? (T)x[e] : (T)0.0f;
      });
    }
  }
  {
    // key features, values, queries and frames of rows c0 .. c0 + ROWS - 1 (zero past n)
    StageRows<T, ROWS, FB, NT> sc;
    StageRows<T, ROWS, DV, NT> sv;
    sc.load(chis, M, c0, 0, n, tid);
    sv.load(vs, DV, c0, 0, n, tid);
    sc.store(sChi, CST, c0, 0, n, tid);
    sv.store(sV, VST, c0, 0, n, tid);
    StageRows<T, ROWS, D, NT> sq;
    sq.load(qs, D, c0, 0, n, tid);
    if constexpr (sizeof(T) == 2) sq.store((f16*)sQ, D + PAD, c0, 0, n, tid);
    else sq.store(sQ, D + PAD, c0, 0, n, tid);
    for (int j = tid; j < ROWS; j += NT) {
      const float rj = (c0 + j < n) ? a.rj[seq + c0 + j] : 0.0f;
      sRj[j] = rj;
      sRat[j] = (c0 + j < n) ? fast_exp2(rj - Rref) : 0.0f;
    }
  }
  __syncthreads();

  f32x16 du[DV / 32];
#pragma unroll
  for (int dt = 0; dt < DV / 32; ++dt) du[dt] = zero16();

  // items 0..31: pair t (rows c0 + t and c0 + 32 NA + t); item 32 r + t
  // (r = 1 .. NA - 1): row c0 + 32 r + t alone.  Row c0 + 32 r + t sees some
  // anchor of the tile iff 32 r + t - 31 < w.
  // one body, compiled for the paired items (0..31) and for the single rows
  auto item = [&](const int it, auto pair_c) {
    constexpr bool pair = decltype(pair_c)::value;
    const int t = it & 31;
    const int rcA = pair ? 0 : it >> 5;                        // chunk of row A relative to kt
    const int iA = c0 + 32 * rcA + t;
    const int iB = c0 + 32 * NA + t;
    const bool okA = iA < n && 32 * rcA + t - 31 < w;          // the row sees the tile
    const bool okB = pair && iB < n && 32 * NA + t - 31 < w;
    if (!okA && !okB) return;
    // row scalars of the (at most two) rows
    const int iAc = min(iA, n - 1), iBc = min(iB, n - 1);
    const float LA = uniform(a.stats[(seq + iAc) * 2]), LB = uniform(a.stats[(seq + iBc) * 2]);
    const float invA = uniform(a.rowstat[(seq + iAc) * 2]), invB = uniform(a.rowstat[(seq + iBc) * 2]);
    const float RA = uniform(okA ? sRj[rcA * 32 + t] : -kNegInf), RB = uniform(okB ? sRj[32 * NA + t] : -kNegInf);
    // dN with the row factor 2^(Rref - R_i) (zero for a row that does not take part)
    const float sbA = uniform(fast_exp2(Rref - RA)), sbB = uniform(fast_exp2(Rref - RB));
    float dNA[DV / 32], dNB[DV / 32];
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) {
      dNA[dt] = tof(gs[(size_t)iAc * DV + dt * 32 + col]) * (invA * sbA);
      dNB[dt] = pair ? tof(gs[(size_t)iBc * DV + dt * 32 + col]) * (invB * sbB) : 0.0f;
    }
    // this lane's row: the one that sees anchor c0 + col
    const bool useB = pair && col > t;
    const int i = useB ? iB : iA;
    const int rc = useB ? NA : rcA;
    const bool valid = (useB ? okB : okA) && (i - c0 - col >= 0) && (i - c0 - col < w);
    typename F::frag pf[FB / 32][F::CSTEPS];
    query_features<T, D, FB>(pf, sQ + (rc * 32 + t) * (D + PAD), sR + col * (D + PAD), sOm, valid, useB ? LB : LA);
    // tails: P^T[j, c] = chi_j . psi_c of chunk kt + rj, times 2^(R_j - Rref), j <= row(c)
    constexpr int NTL = NA + 1;
    typename F::frag ppf[NTL][F::CSTEPS];
    const int ntl = okB ? NTL : rcA + 1;                        // tails any lane needs
#pragma unroll
    for (int rj = 0; rj < NTL; ++rj) {
      if (rj >= ntl) {
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp) ppf[rj][sp] = F::zero();
        continue;
      }
      f32x16 accP = zero16();
      const T* chirow = sChi + (rj * 32 + col) * CST;
#pragma unroll
      for (int pt = 0; pt < FB / 32; ++pt)
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp)
          accP = F::mma(F::ldc(chirow, pt * 32, sp, h), pf[pt][sp], accP);
      const int lim = rj < rc ? 31 : (rj == rc ? t : -1);      // last token of chunk rj this lane's row sees
      const float* sRh = sRat + rj * 32 + 4 * h;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 r4 = *(const f32x4*)(sRh + 8 * g);
#pragma unroll
        for (int e = 0; e < 4; ++e) accP[4 * g + e] *= (8 * g + 4 * h + e <= lim) ? r4[e] : 0.0f;
      }
#pragma unroll
      for (int sp = 0; sp < F::CSTEPS; ++sp) ppf[rj][sp] = F::cfrag(accP, sp);
    }
    // two 32-wide d slices per step (two independent matrix-core chains);
    // registers <-> anchor crow(v, h), which takes its row's frame and dN
    constexpr int G = DV / 32 >= 2 ? 2 : 1;
#pragma unroll
    for (int d0 = 0; d0 < DV / 32; d0 += G) {
      no_hoist();
      f32x16 accA[G];
#pragma unroll
      for (int g = 0; g < G; ++g) accA[g] = zero16();
#pragma unroll
      for (int pt = 0; pt < FB / 32; ++pt)
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp)
#pragma unroll
          for (int g = 0; g < G; ++g)
            accA[g] = F::mma(pf[pt][sp], F::ldc(sMt + ((d0 + g) * 32 + col) * (FB + PAD), pt * 32, sp, h), accA[g]);
#pragma unroll
      for (int rj = 0; rj < NTL; ++rj) {
        if (rj >= ntl) continue;
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp)
#pragma unroll
          for (int g = 0; g < G; ++g)
            accA[g] = F::mma(ppf[rj][sp], F::tld_crow(sV, VST, rj * 32, sp, (d0 + g) * 32), accA[g]);
      }
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int v = 0; v < 16; ++v) du[d0 + g][v] += accA[g][v] * ((pair && crow(v, h) > t) ? dNB[d0 + g] : dNA[d0 + g]);
    }
  };
#pragma unroll 1
  for (int it = wv; it < 32; it += NW) item(it, std::true_type{});
#pragma unroll 1
  for (int it = 32 + wv; it < 32 * NA; it += NW) item(it, std::false_type{});
  reduce_waves<DV / 32>(du, (float*)smem, wv, NW);
  if (wv == 0) {
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int c = c0 + crow(v, h);
        if (c >= n) continue;
        if constexpr (M / FB == 1) ((T*)a.du)[(seq + c) * DV + dt * 32 + col] = (T)du[dt][v];
        else a.du32[(((size_t)fb * a.BH + bh) * n + c) * DV + dt * 32 + col] = du[dt][v];
      }
  }
}

// ---------------------------------------------------------------------------
// k_bwd_dqdr: per (row i, anchor c), dA = dN_i (*) u_c and
//   dpsi[p, c] = sb_i (M_b dA_c + dZ_i a_b)[p] + sum_{j <= i} 2^(R_j - R_i) chi_j[p] (v_j . dA_c + dZ_i)
//   dell = dpsi (*) psi,  s_c = sum_p dell[p, c]
//   dz_c = Omega^T dell_c - s_c z_c  ->  dr_c += dz_c (*) q_i,  dq_i += dz_c (*) r_c
// dr stays in registers (regs <-> anchor, lanes <-> D); each row's dq over this
// tile is complete in one wave and goes to slot (chunk of i) - (tile) of dq32.
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M, int NA>
__global__ __launch_bounds__(64 * 8) void k_bwd_dqdr(BwdArgs a) {
  using F = MF<T>;
  using C = AsCfg<T, D, DV, M, NA>;
  constexpr int PAD = C::PAD, FB = C::FB, NW = C::NW;
  constexpr int NT = 64 * NW;
  constexpr int S = M * DV + M;
  constexpr int NS = NA + 1;
  static_assert(C::BYTES <= 160 * 1024, "dqdr LDS budget");
  __shared__ __align__(16) char smem[C::BYTES];
  T* sOm = (T*)(smem + C::oOm);
  T* sMp = (T*)(smem + C::oM);
  T* sChi = (T*)(smem + C::oChi);
  T* sV = (T*)(smem + C::oV);
  T* sQ = (T*)(smem + C::oQ);
  T* sR = (T*)(smem + C::oR);
  T* sU = (T*)(smem + C::oU);
  float* sRj = (float*)(smem + C::oRj);
  float* sA = (float*)(smem + C::oA);
  float* sRat = (float*)(smem + C::oRat);

  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  float* sDN = (float*)(smem + C::oW) + wv * (DV + 32);
  float* sSc = sDN + DV;
  const int2 gxy = xcd_grid_xy();
  const int kt = gxy.x, bh = gxy.y, hh = bh % a.H, n = a.n, nch = a.nch, fb = blockIdx.z;
  const int c0 = kt * 32, w = a.w;
  const size_t seq = (size_t)bh * n;
  const T* qs = (const T*)a.q + seq * D;
  const T* vs = (const T*)a.v + seq * DV;
  const T* rs_ = (const T*)a.r + seq * D;
  const T* us = (const T*)a.u + seq * DV;
  const T* gs = (const T*)a.dout + seq * DV;
  const T* chis = (const T*)a.chi + seq * M + fb * FB;
  const T* omq_h = (const T*)a.omq + (size_t)hh * M * D;

  T* sOb = (T*)(smem + C::oOb);
  {
    // Omega (float32) once for both LDS copies, r and u of the anchor tile
    StageRows<float, FB, D, NT> so;
    StageRows<T, 32, D, NT> sr;
    StageRows<T, 32, DV, NT> su;
    so.load(a.omega + ((size_t)hh * M + (size_t)fb * FB) * D, D, 0, 0, FB, tid);
    sr.load(rs_, D, c0, 0, n, tid);
    su.load(us, DV, c0, 0, n, tid);
    so.store(sOb, D + C::TPD, 0, 0, FB, tid);
    if constexpr (sizeof(T) == 2) {
      so.store((f16*)sOm, D + PAD, 0, 0, FB, tid, kLog2e);
      sr.store((f16*)sR, C::RST, c0, 0, n, tid);
      su.store((f16*)sU, DV + PAD, c0, 0, n, tid);
    } else {
      so.store(sOm, D + PAD, 0, 0, FB, tid, kLog2e);
      sr.store(sR, C::RST, c0, 0, n, tid);
      su.store(sU, DV + PAD, c0, 0, n, tid);
    }
  }
  f32x16 dr[D / 32];
#pragma unroll
  for (int Dt = 0; Dt < D / 32; ++Dt) dr[Dt] = zero16();
  const int ch_end = min(nch - 1, (c0 + 30 + w) / 32);

#pragma unroll 1
  for (int ch = kt; ch <= ch_end; ++ch) {
    const int s0 = ch * 32;
    const bool has_bnd = ch > 0;
    const float Rexb = a.rex[(size_t)bh * (nch + 1) + ch];
    // reference frame of the chunk's rows: the boundary frame (the first chunk,
    // whose boundary state is zero, takes R of its first row); with it
    //   dpsi = 2^(Rref - R_i) [M_b dA + dZ a_b + sum_{j <= i} 2^(R_j - Rref) chi_j (v_j . dA + dZ)]
    // and the row factor 2^(Rref - R_i) goes into dN and dZ once per row
    const float Rref = uniform(has_bnd ? Rexb : a.rj[seq + s0]);
    {
      // the chunk's global loads, each batch issued in full before its LDS
      // stores (float32 inputs: the state in two halves, the second with
      // the chunk rows; bf16 inputs: the bf16 state at once)
      constexpr int FH = FB / 2;
      StageState<FH, DV, NT, false> sm;
      StageRows<T, FB, DV, NT> sm16;
      const float* bst = a.states + ((size_t)bh * nch + ch) * S;
      float av = 0.0f;
      if (has_bnd) {
        if constexpr (sizeof(T) == 2) sm16.load((const T*)a.states16 + (((size_t)bh * nch + ch) * M + (size_t)fb * FB) * DV, DV, 0, 0, FB, tid);
        else sm.load(bst + (size_t)fb * FB * DV, tid);
        if (tid < FB) av = bst[(size_t)M * DV + fb * FB + tid];
      }
      __syncthreads();
      auto put = [&](int p0) {
        return [&, p0](int p, int d0, const f32x4& x) {
#pragma unroll
          for (int e = 0; e < 4; ++e) sMp[(p0 + p) * (DV + PAD) + d0 + e] = has_bnd ? (T)x[e] : (T)0.0f;
        };
      };
      // the first chunk stages a zero boundary state, so that the boundary
      // product below needs no branch (its accumulator chain then starts
      // from an inline zero and the sweep keeps more registers)
      if constexpr (sizeof(T) == 2) {
        sm16.store(sMp, DV + PAD, has_bnd ? 0 : FB, 0, FB, tid);   // rows outside [0, FB): zero
      } else {
        sm.store(tid, put(0));
        if (has_bnd) sm.load(bst + (size_t)(fb * FB + FH) * DV, tid);
      }
      if (tid < FB) sA[tid] = av;
      if constexpr (sizeof(T) == 2) {
        // bf16: a_b rides in the padding of M_b's row p as one more k-step of
        // the boundary product, (a_hi, a_hi, a_lo, 0, ...) against the row's
        // (dZ_hi, dZ_lo, dZ_hi, 0, ...): a_b dZ to about 16 bits
        if (tid < FB) {
          const bf16 ah = (bf16)av, al = (bf16)(av - (float)ah), z = (bf16)0.0f;
          *(bf16x8*)(sMp + tid * (DV + PAD) + DV) = bf16x8{ah, ah, al, z, z, z, z, z};
        }
      }
      StageRows<T, 32, FB, NT> sc;
      StageRows<T, 32, DV, NT> sv;
      StageRows<T, 32, D, NT> sq;
      sc.load(chis, M, s0, 0, n, tid);
      sv.load(vs, DV, s0, 0, n, tid);
      sq.load(qs, D, s0, 0, n, tid);
      const float rjv = (tid < 32) ? a.rj[seq + min(s0 + tid, n - 1)] : 0.0f;
      if constexpr (sizeof(T) != 2) sm.store(tid, put(FH));
      sc.store(sChi, C::CST, s0, 0, n, tid);
      sv.store(sV, C::VST, s0, 0, n, tid);
      if constexpr (sizeof(T) == 2) sq.store((f16*)sQ, D + PAD, s0, 0, n, tid);
      else sq.store(sQ, D + PAD, s0, 0, n, tid);
      if (tid < 32) {
        sRj[tid] = (s0 + tid < n) ? rjv : 0.0f;
        sRat[tid] = (s0 + tid < n) ? fast_exp2(rjv - Rref) : 0.0f;
      }
    }
    __syncthreads();

    // upstream-gradient rows are fetched one row ahead
    constexpr int NG = (DV + 63) / 64;
    float gpre[NG];
    auto load_g = [&](int t) {
      const size_t i = (size_t)min(s0 + t, n - 1);
#pragma unroll
      for (int e = 0; e < NG; ++e) gpre[e] = (e * 64 + l < DV) ? tof(gs[i * DV + e * 64 + l]) : 0.0f;
    };
    load_g(wv);
#pragma unroll 1
    for (int t = wv; t < 32; t += NW) {
      float gv[NG];
#pragma unroll
      for (int e = 0; e < NG; ++e) gv[e] = gpre[e];
      if (t + NW < 32) load_g(t + NW);
      const int i = s0 + t;
      if (i >= n || i < c0 || i - c0 > w + 30) continue;
      __builtin_amdgcn_iglp_opt(0);             // interleave the matrix-core and LDS streams
      const float Li = uniform(a.stats[(seq + i) * 2]);
      const float inv = uniform(a.rowstat[(seq + i) * 2]);
      const float dZ = uniform(a.rowstat[(seq + i) * 2 + 1]);
      const float Ri = uniform(sRj[t]);
      const float sbr = uniform(fast_exp2(Rref - Ri));
      const float dZr = dZ * sbr;
      const float invr = inv * sbr;
#pragma unroll
      for (int e = 0; e < NG; ++e)
        if (e * 64 + l < DV) sDN[e * 64 + l] = gv[e] * invr;
      const T* qrow = sQ + t * (D + PAD);
      float qD[D / 32];
#pragma unroll
      for (int Dt = 0; Dt < D / 32; ++Dt)
        qD[Dt] = sizeof(T) == 2 ? (float)((const f16*)qrow)[Dt * 32 + col] : tof(qrow[Dt * 32 + col]);
      wave_lds_sync();
      const int c = c0 + col;
      const bool valid = (i - c >= 0) && (i - c < w);
      // psi only scales dpsi here: f16 fragments (bf16 inputs)
      using PF = typename std::conditional<sizeof(T) == 2, f16x8, typename F::frag>::type;
      PF pf[FB / 32][F::CSTEPS];
      query_features<T, D, FB, PF>(pf, qrow, sR + col * (C::RST), sOm, valid, Li);
      // dA^T fragments: lanes <-> anchor, natural d order
      const T* urow = sU + col * (DV + PAD);
      typename F::frag daf[DV / F::KS];
#pragma unroll
      for (int s = 0; s < DV / F::KS; ++s) {
        const int k0 = s * F::KS + h * F::KPL;
        if constexpr (sizeof(T) == 2) {
          const f16x8 uf = *(const f16x8*)((const f16*)urow + k0);
          const f32x4 d0 = *(const f32x4*)(sDN + k0), d1 = *(const f32x4*)(sDN + k0 + 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            daf[s][e] = (bf16)__builtin_fmaf((float)uf[e], d0[e], 0.0f);   // one mixed-precision FMA
            daf[s][4 + e] = (bf16)__builtin_fmaf((float)uf[4 + e], d1[e], 0.0f);
          }
        } else {
          daf[s] = F::ld(urow, k0) * sDN[k0];
        }
      }
      // Q^T[j, c] = (v_j . dA_c + dZ_i) 2^(R_j - Rref), j <= i  (regs <-> j, lanes <-> anchor;
      // dA and dZ carry the row factor)
      f32x16 accQ = zero16();
#pragma unroll
      for (int s = 0; s < DV / F::KS; ++s)
        accQ = F::mma(F::ld(sV + col * C::VST, s * F::KS + h * F::KPL), daf[s], accQ);
      float sj[16];
      masked_ratios(sj, sRat, t);
#pragma unroll
      for (int v = 0; v < 16; ++v) accQ[v] = (accQ[v] + dZr) * sj[v];
      typename F::frag qqf[F::CSTEPS];
#pragma unroll
      for (int sp = 0; sp < F::CSTEPS; ++sp) qqf[sp] = F::cfrag(accQ, sp);
      // the boundary product's k-step for dZ a_b (bf16; lanes of the upper half zero)
      typename F::frag zb = F::zero();
      if constexpr (sizeof(T) == 2) {
        const bf16 zh = (bf16)dZr, zl = (bf16)(dZr - (float)zh);
        if (h == 0) { zb[0] = zh; zb[1] = zl; zb[2] = zh; }
      }
      // dell = dpsi (*) psi (derivative with respect to the natural-log feature)
      typename F::frag dlf[FB / 32][F::CSTEPS];
      float sc = 0.0f;
#pragma unroll
      for (int pt = 0; pt < FB / 32; ++pt) {
        no_hoist();
        // boundary part M_b dA_c + dZ_i a_b (row factor in dA, dZ), zero in the first chunk
        f32x16 dps = zero16();
#pragma unroll
        for (int s = 0; s < DV / F::KS; ++s)
          dps = F::mma(F::ld(sMp + (pt * 32 + col) * (DV + PAD), s * F::KS + h * F::KPL), daf[s], dps);
        if constexpr (sizeof(T) == 2) {
          dps = F::mma(*(const bf16x8*)(sMp + (pt * 32 + col) * (DV + PAD) + DV), zb, dps);
        } else {
          const float* sAh = sA + pt * 32 + 4 * h;
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x4 av = *(const f32x4*)(sAh + 8 * g);
#pragma unroll
            for (int e = 0; e < 4; ++e) dps[4 * g + e] = __builtin_fmaf(dZr, av[e], dps[4 * g + e]);
          }
        }
        // chi^T rows p, k = token j in crow order (chi stored [j][sigma(p)])
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp) {
          typename F::frag cf;
          if constexpr (sizeof(T) == 2) {
            const int g = l >> 4, s4 = l & 15;
            const int pcol = F::sigma(pt * 32 + 16 * (g & 1) + 4 * (s4 & 3));
            bf16x4 x0 = lds_tr4(sChi + (16 * sp + 4 * h + (s4 >> 2)) * (C::CST) + pcol);
            bf16x4 x1 = lds_tr4(sChi + (16 * sp + 8 + 4 * h + (s4 >> 2)) * (C::CST) + pcol);
            cf = cat44(x0, x1);
          } else {
            cf = sChi[crow(sp, h) * (C::CST) + pt * 32 + col];
          }
          dps = F::mma(cf, qqf[sp], dps);
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) dps[v] = __builtin_fmaf(fel(pf[pt][v / F::KPL], v % F::KPL), dps[v], 0.0f);
        // s_c sums dlambda as rounded for dz's matrix product: the two terms of
        // dz = sum_p dlambda_p (Omega_p - z) partly cancel, and a rounding in
        // one of them only would be amplified by that
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp) {
          dlf[pt][sp] = F::cfrag(dps, sp);
          sc = add_elems(dlf[pt][sp], sc);
        }
      }
      sc = half_swap_add(sc);
      if (h == 0) sSc[col] = valid ? sc : 0.0f;
      wave_lds_sync();
      // dz[c, D] (regs <-> anchor, lanes <-> D)
      float* dqo = a.dq32 + ((((size_t)fb * NS + (ch - kt)) * a.BH + bh) * n + i) * D;
#pragma unroll
      for (int Dt = 0; Dt < D / 32; ++Dt) {
        no_hoist();
        f32x16 dz = zero16();
#pragma unroll
        for (int pt = 0; pt < FB / 32; ++pt)
#pragma unroll
          for (int sp = 0; sp < F::CSTEPS; ++sp)
            dz = F::mma(dlf[pt][sp], F::tld_crow(sOb, D + C::TPD, pt * 32, sp, Dt * 32), dz);
        float rv[16];
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp) {
          if constexpr (sizeof(T) == 2) {
            const f16x8 rf = tld_crow_f16((const f16*)sR, C::RST, 0, sp, Dt * 32);
#pragma unroll
            for (int e = 0; e < 8; ++e) rv[8 * sp + e] = (float)rf[e];
          } else {
            rv[sp] = F::tld_crow(sR, C::RST, 0, sp, Dt * 32);
          }
        }
        const float qd = qD[Dt];
        const float* sch = sSc + 4 * h;
        float dqs = 0.0f;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 s4 = *(const f32x4*)(sch + 8 * g);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int v = 4 * g + e;
            const float dzz = dz[v] - s4[e] * qd * rv[v];
            dqs += dzz * rv[v];
            dr[Dt][v] += dzz * qd;
          }
        }
        dqs = half_swap_add(dqs);
        if (h == 0) dqo[Dt * 32 + col] = dqs;
      }
    }
  }
  reduce_waves<D / 32>(dr, (float*)smem, wv, NW);
  if (wv == 0) {
#pragma unroll
    for (int Dt = 0; Dt < D / 32; ++Dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int c = c0 + crow(v, h);
        if (c >= n) continue;
        if constexpr (C::NFB == 1) ((T*)a.dr)[(seq + c) * D + Dt * 32 + col] = (T)dr[Dt][v];
        else a.dr32[(((size_t)fb * a.BH + bh) * n + c) * D + Dt * 32 + col] = dr[Dt][v];
      }
  }
}

// dq of every row: sum over feature blocks and over the anchor tiles that
// processed it (tile k = chunk(i) - slot, processed iff k >= 0 and i - 32k <= w + 30)
template <typename T>
__global__ __launch_bounds__(256) void k_bwd_final_dq(const float* __restrict__ src, T* __restrict__ dst,
                                                      int BH, int n, int D, int nfb, int NS, int w) {
  // four consecutive elements of one row per thread (D is a multiple of 4)
  const size_t count = (size_t)BH * n * D;
  const size_t idx = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (idx >= count) return;
  const int i = (int)((idx / D) % n);
  const int bi = i >> 5;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int fb = 0; fb < nfb; ++fb)
    for (int s = 0; s < NS; ++s) {
      const int k = bi - s;
      if (k < 0 || i - 32 * k > w + 30) continue;
      acc += *(const f32x4*)(src + ((size_t)fb * NS + s) * count + idx);
    }
  typedef T V4 __attribute__((ext_vector_type(4)));
  V4 y;
#pragma unroll
  for (int e = 0; e < 4; ++e) y[e] = (T)acc[e];
  *(V4*)(dst + idx) = y;
}

// ---------------------------------------------------------------------------
// k_bwd_state: state sweep of one chunk b, one wave per 32-feature tile.
// With dM^(i)[p, d] = sum_c psi_icp dA_ic[d] and da^(i)[p] = dZ_i sum_c psi_icp,
// the rows are walked in reverse with the running (frame R_t) matrices
//   F_t = dM^(t) + 2^(R_t - R_{t+1}) F_{t+1},   f_t likewise from da,
// i.e. F_t = sum_{i >= t in the chunk} 2^(R_t - R_i) dM^(i).  They give
//   intra dchi_t = F_t v_t + f_t      intra dv_t = F_t^T chi_t
//   GB_b = sum_i sb_i dM^(i) = 2^(Rex_b - R_s0) F_s0,   gb_b = 2^(Rex_b - R_s0) f_s0.
// The query features are formed with the (row, anchor) pair in registers
// (lanes <-> feature p): L[c, p] = sum_D r_c[D] (q_i[D] Omega[p, D]), so the
// wave's Omega tile is scaled by q_i once per row and multiplies the anchors'
// r rows straight from LDS; |q_i (*) r_c|^2 comes from a per-chunk table built
// with the matrix cores (q^2 against r^2, split hi + lo in bf16).
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M, int NA>
struct StCfg {
  static constexpr int PAD = MF<T>::PAD;
  static constexpr int FB = M < 128 ? M : 128;
  static constexpr int NFB = M / FB;
  static constexpr int NW = FB / 32;
  static constexpr int AW = 32 * NA;                 // anchor offsets i - c per row
  static constexpr int WIN = 32 + AW - 1;            // anchor window rows of a chunk
  static constexpr int NT32 = (WIN + 31) / 32;
  static constexpr int RB = 2;                       // rows per intra-dv flush (two: the
                                                     // room goes to full-rate u rows below)
  static constexpr int ES = sizeof(T);
  static constexpr int a16(int x) { return (x + 15) & ~15; }
  static constexpr int oR = 0;
  static constexpr int oU = oR + a16(32 * NT32 * (D + PAD) * ES);
  // bytes after the u window (rows of pitch DV + tp)
  static constexpr int tail(int tp) {
    return a16(WIN * (DV + tp) * ES) + a16(32 * (FB + PAD) * ES) + a16(32 * AW * 4) + 2 * a16(32 * 4) +
           a16(NW * D * ES) + a16(NW * RB * DV * 4);
  }
  // two workgroups per CU up to two anchor tiles per row (w <= 64); wider
  // windows stage up to 159 anchor rows and run one workgroup per CU
  static constexpr int LDS_CAP = NA <= 2 ? 80 * 1024 : 160 * 1024;
  static constexpr int MINB = NA <= 2 ? 2 : 1;
  // full-rate transposing reads of u when the budget allows
  static constexpr int TP = (oU + tail(tr_pad<T, DV>()) <= LDS_CAP || sizeof(T) != 2) ? tr_pad<T, DV>() : 16;
  static constexpr int oChi = oU + a16(WIN * (DV + TP) * ES);
  static constexpr int oNz = oChi + a16(32 * (FB + PAD) * ES);
  static constexpr int oRj = oNz + a16(32 * AW * 4);
  static constexpr int oL = oRj + a16(32 * 4);
  static constexpr int oQ = oL + a16(32 * 4);
  static constexpr int oDv = oQ + a16(NW * D * ES);
  static constexpr int BYTES = oDv + a16(NW * RB * DV * 4);
};

template <typename T> LS_DEV void ld4f(const T* p, float (&x)[4]) {
  if constexpr (sizeof(T) == 2) {
    bf16x4 b = *(const bf16x4*)p;
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = (float)b[e];
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = p[e];
  }
}

// squared fragment, split into hi + lo parts of the operand type
template <typename T> LS_DEV void sq_split(const typename MF<T>::frag& x, typename MF<T>::frag& hi,
                                           typename MF<T>::frag& lo) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float s = fel(x, e) * fel(x, e);
      hi[e] = (bf16)s;
      lo[e] = (bf16)(s - (float)hi[e]);
    }
  } else {
    hi = x * x;
    lo = 0.0f;
  }
}

template <typename T, int D, int DV, int M, int NA>
__global__ __launch_bounds__(256, (NA <= 2 ? 2 : 1)) void k_bwd_state(BwdArgs a) {
  using F = MF<T>;
  using C = StCfg<T, D, DV, M, NA>;
  constexpr int PAD = C::PAD, FB = C::FB, WIN = C::WIN, NW = C::NW, AW = C::AW, RB = C::RB;
  constexpr int NT = 64 * NW;
  static_assert(C::BYTES <= C::LDS_CAP, "state LDS budget");
  __shared__ __align__(16) char smem[C::BYTES];
  T* sR = (T*)(smem + C::oR);
  T* sU = (T*)(smem + C::oU);
  T* sChi = (T*)(smem + C::oChi);
  float* sNz = (float*)(smem + C::oNz);        // [t][i - c]: -|z|^2 log2e / 2 - L_i, -inf if not a pair
  float* sRj = (float*)(smem + C::oRj);
  float* sL = (float*)(smem + C::oL);
  float* sDv = (float*)(smem + C::oDv);        // [wave][row % RB][d] intra dv partials

  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  T* sQ = (T*)(smem + C::oQ) + wv * D;
  const int2 gxy = xcd_grid_xy();
  const int cb = gxy.x, bh = gxy.y, hh = bh % a.H, n = a.n, nch = a.nch, fb = blockIdx.z;
  const int s0 = cb * 32;
  const int wb = s0 - (AW - 1);                // window row 0 = anchor s0 - (AW - 1)
  const int tlast = min(31, n - 1 - s0);
  const size_t seq = (size_t)bh * n;
  const T* qs = (const T*)a.q + seq * D;
  const T* vs = (const T*)a.v + seq * DV;
  const T* rs_ = (const T*)a.r + seq * D;
  const T* us = (const T*)a.u + seq * DV;
  const T* gs = (const T*)a.dout + seq * DV;
  const T* omq_h = (const T*)a.omq + (size_t)hh * M * D;
  const float Rexb = a.rex[(size_t)bh * (nch + 1) + cb];
  const int w = a.w;
  const int pw = fb * FB + wv * 32;            // first feature of this wave's tile

  {
    // every global load of the window first, then the LDS stores
    StageRows<T, 32 * C::NT32, D, NT> sr;
    StageRows<T, WIN, DV, NT> su;
    StageRows<T, 32, FB, NT> sc;
    sr.load(rs_, D, wb, 0, n, tid);
    su.load(us, DV, wb, 0, n, tid);
    sc.load((const T*)a.chi + seq * M + fb * FB, M, s0, 0, n, tid);   // key features of the chunk
    const float lv = (tid < 32) ? a.stats[(seq + min(s0 + tid, n - 1)) * 2] : 0.0f;
    const float rjv = (tid < 32) ? a.rj[seq + min(s0 + tid, n - 1)] : 0.0f;
    if constexpr (sizeof(T) == 2) sr.store((f16*)sR, D + PAD, wb, 0, n, tid);
    else sr.store(sR, D + PAD, wb, 0, n, tid);
    su.store(sU, DV + C::TP, wb, 0, n, tid);
    sc.store(sChi, FB + PAD, s0, 0, n, tid);
    if (tid < 32) {
      sL[tid] = (s0 + tid < n) ? lv : 0.0f;
      sRj[tid] = (s0 + tid < n) ? rjv : 0.0f;
    }
  }
  __syncthreads();
  // the |z|^2 table
  {
    for (int kt = wv; kt < C::NT32; kt += NW) {
      // C[t][wi] = sum_D q_{s0+t}[D]^2 r_{wb+wi}[D]^2   (regs <-> t, lanes <-> window row)
      f32x16 acc = zero16();
      const bool vi = s0 + col < n;
      const T* qrow = qs + (size_t)(vi ? s0 + col : 0) * D;
      const T* rrow = sR + (32 * kt + col) * (D + PAD);
#pragma unroll 2
      for (int s = 0; s < D / F::KS; ++s) {
        const int k0 = s * F::KS + h * F::KPL;
        typename F::frag qf = vi ? F::ld(qrow, k0) : F::zero();
        typename F::frag qh, ql, rh, rl;
        sq_split<T>(qf, qh, ql);
        if constexpr (sizeof(T) == 2) {
          // bf16 inputs: r is held as f16 (exact for bf16 values in the normal range)
          const f16x8 r16 = *(const f16x8*)((const f16*)rrow + k0);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float x = (float)r16[e], sq = x * x;
            rh[e] = (bf16)sq;
            rl[e] = (bf16)(sq - (float)rh[e]);
          }
        } else {
          sq_split<T>(F::ld(rrow, k0), rh, rl);
        }
        acc = F::mma(qh, rh, acc);
        if constexpr (sizeof(T) == 2) {
          acc = F::mma(qh, rl, acc);
          acc = F::mma(ql, rh, acc);
        }
      }
      const int wi = 32 * kt + col;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int t = crow(v, h);
        const int dl = t - wi + AW - 1;            // i - c
        if (dl >= 0 && dl < AW) {
          const bool ok = dl < w && wb + wi >= 0 && s0 + t < n;
          sNz[t * AW + dl] = ok ? -0.5f * kLog2e * acc[v] - sL[t] : kNegInf;
        }
      }
    }
  }
  // this wave's Omega tile (log2e-scaled) as B operands, resident in registers
  // (bf16 inputs: f16 copies of Omega*log2 e, q and r; the logits use the f16 matrix cores)
  using OF = typename std::conditional<sizeof(T) == 2, f16x8, float>::type;
  OF omf[D / F::KS];
#pragma unroll
  for (int s = 0; s < D / F::KS; ++s) {
    const int k0 = s * F::KS + h * F::KPL;
    if constexpr (sizeof(T) == 2) {
      omf[s] = *(const f16x8*)((const f16*)a.omh + ((size_t)hh * M + pw + col) * D + k0);
    } else {
      omf[s] = F::ld(omq_h + (size_t)(pw + col) * D, k0);
    }
  }
  __syncthreads();

  f32x16 Fm[DV / 32];
#pragma unroll
  for (int dt = 0; dt < DV / 32; ++dt) Fm[dt] = zero16();
  float fpart = 0.0f;                          // f[p = col], partial over this half's anchors

  // the rows' q, dout, v and statistics are fetched one row ahead
  constexpr int QE = (D + 63) / 64;
  T qn[QE], gn[DV / 32], vn[DV / 32];
  float invn, dZn;
  auto fetch = [&](int t) {
    const size_t i = (size_t)(s0 + t);
#pragma unroll
    for (int e = 0; e < QE; ++e) qn[e] = (e * 64 + l < D) ? qs[i * D + e * 64 + l] : (T)0.0f;
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) {
      gn[dt] = gs[i * DV + dt * 32 + col];
      vn[dt] = vs[i * DV + dt * 32 + col];
    }
    invn = a.rowstat[(seq + i) * 2];
    dZn = a.rowstat[(seq + i) * 2 + 1];
  };
  fetch(tlast);
#pragma unroll 1
  for (int t = tlast; t >= 0; --t) {
    const float inv = uniform(invn);
    const float dZ = uniform(dZn);
    const float fr = uniform(t < tlast ? fast_exp2(sRj[t] - sRj[t + 1]) : 1.0f);
#pragma unroll
    for (int e = 0; e < QE; ++e)
      if (e * 64 + l < D) {
        if constexpr (sizeof(T) == 2) ((f16*)sQ)[e * 64 + l] = (f16)(float)qn[e];
        else sQ[e * 64 + l] = qn[e];
      }
    float dN[DV / 32], vv[DV / 32];
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) {
      dN[dt] = tof(gn[dt]) * inv;
      vv[dt] = tof(vn[dt]);
    }
    if (t > 0) fetch(t - 1);
    const int i = s0 + t;
    wave_lds_sync();
    // logits L[c, p] of the row's anchor tiles (regs <-> anchor c = i - 32an - crow)
    f32x16 acc[NA];
#pragma unroll
    for (int an = 0; an < NA; ++an) acc[an] = zero16();
#pragma unroll
    for (int s = 0; s < D / F::KS; ++s) {
      const int k0 = s * F::KS + h * F::KPL;
      if constexpr (sizeof(T) == 2) {
        const f16x8 bq = omf[s] * *(const f16x8*)((const f16*)sQ + k0);
#pragma unroll
        for (int an = 0; an < NA; ++an)
          acc[an] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
              *(const f16x8*)((const f16*)sR + (t + AW - 1 - 32 * an - col) * (D + PAD) + k0), bq, acc[an], 0, 0, 0);
      } else {
        const float bq = omf[s] * F::ld(sQ, k0);
#pragma unroll
        for (int an = 0; an < NA; ++an)
          acc[an] = F::mma(F::ld(sR + (t + AW - 1 - 32 * an - col) * (D + PAD), k0), bq, acc[an]);
      }
    }
    // psi = 2^(L + bias); bias -inf outside the window
    typename F::frag pf[NA][F::CSTEPS];
    float ps = 0.0f;
#pragma unroll
    for (int an = 0; an < NA; ++an) {
      const float* brow = sNz + t * AW + 32 * an + 4 * h;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 b4 = *(const f32x4*)(brow + 8 * g);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[an][4 * g + e] = fast_exp2(acc[an][4 * g + e] + b4[e]);
      }
      // f sums the features exactly as rounded for F's matrix product: the two
      // cancel in dchi = F v + f (the output is a ratio), and a rounding in
      // one of them only would be amplified by that cancellation
#pragma unroll
      for (int sp = 0; sp < F::CSTEPS; ++sp) {
        pf[an][sp] = F::cfrag(acc[an], sp);
        ps = add_elems(pf[an][sp], ps);
      }
    }
    if (fr != 1.0f) {
      fpart *= fr;
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt) Fm[dt] *= fr;
    }
    fpart += dZ * ps;
    // F <- 2^(R_t - R_{t+1}) F + (sum_c psi_c u_c^T) diag(dN)
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) {
      f32x16 y = zero16();
#pragma unroll
      for (int an = 0; an < NA; ++an) {
        auto rmap = [&](int ar) { return t + AW - 1 - 32 * an - ar; };
#pragma unroll
        for (int sp = 0; sp < F::CSTEPS; ++sp)
          y = F::mma(pf[an][sp], F::tld_crow_map(sU, DV + C::TP, sp, dt * 32, rmap), y);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) Fm[dt][v] += y[v] * dN[dt];
    }
    // intra dchi_t[p] = F_t[p, :] . v_t + f_t[p]  (p of register col >> 1)
    float X[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float x = 0.0f;
#pragma unroll
      for (int dt = 0; dt < DV / 32; ++dt) x += Fm[dt][v] * vv[dt];
      X[v] = x;
    }
    const float xs = half_reduce16(X);
    const int pl = crow(col >> 1, h);
    const float ft = __shfl(half_swap_add(fpart), pl);
    if ((col & 1) == 0) a.dchi[(seq + i) * M + pw + pl] = xs + ft;
    // intra dv_t[d] = sum_p chi_t[p] F_t[p, d]  (this wave's p tile; summed over waves below)
    float chv[16];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float c4[4];
      ld4f<T>(sChi + t * (FB + PAD) + F::sigma(wv * 32 + 8 * g + 4 * h), c4);
#pragma unroll
      for (int e = 0; e < 4; ++e) chv[4 * g + e] = c4[e];
    }
#pragma unroll
    for (int dt = 0; dt < DV / 32; ++dt) {
      float x = 0.0f;
#pragma unroll
      for (int v = 0; v < 16; ++v) x += chv[v] * Fm[dt][v];
      x = half_swap_add(x);
      if ((dt & 1) == h) sDv[(wv * RB + t % RB) * DV + dt * 32 + col] = x;
    }
    if (t % RB == 0) {
      __syncthreads();
      float* dvin = a.dvin + ((size_t)fb * a.BH + bh) * n * DV;
      for (int idx = tid; idx < RB * DV; idx += NT) {
        const int rr = idx / DV, d = idx % DV;
        if (t + rr <= tlast) {
          float x = 0.0f;
#pragma unroll
          for (int ww = 0; ww < NW; ++ww) x += sDv[(ww * RB + rr) * DV + d];
          dvin[(size_t)(s0 + t + rr) * DV + d] = x;
        }
      }
      __syncthreads();
    }
  }
  // ---- GB (frame Rex_b) and gb ----
  constexpr int S = M * DV + M;
  float* g = a.gst + ((size_t)bh * nch + cb) * S;
  const float fac = fast_exp2(Rexb - sRj[0]);  // 0 for the first chunk (Rex_0 = -inf)
#pragma unroll
  for (int dt = 0; dt < DV / 32; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) g[(size_t)(pw + crow(v, h)) * DV + dt * 32 + col] = Fm[dt][v] * fac;
  const float ft = half_swap_add(fpart);
  if (h == 0) g[(size_t)M * DV + pw + col] = ft * fac;
}

// ---------------------------------------------------------------------------
// reverse exclusive scan:  Ghat_b = GB_{b+1} + 2^(Rex_{b+1} - Rex_{b+2}) Ghat_{b+1},
// Ghat_{nch-1} = 0  (frame of Ghat_b: Rex_{b+1}, the running key max at the end
// of chunk b).  In place, element-parallel, sequential over chunks.
// ---------------------------------------------------------------------------
template <int S>
__global__ __launch_bounds__(256) void k_bwd_revscan(BwdArgs a) {
  constexpr int PF = 8;
  const int bh = blockIdx.y;
  const int i4 = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (i4 >= S) return;
  const int nch = a.nch;
  float* g = a.gst + (size_t)bh * nch * S;
  const float* rx = a.rex + (size_t)bh * (nch + 1);
  f32x4 run = {0.f, 0.f, 0.f, 0.f};
  for (int b1 = nch - 1; b1 >= 0; b1 -= PF) {
    f32x4 x[PF];
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      int b = b1 - e;
      x[e] = (b >= 0) ? *(const f32x4*)(g + (size_t)b * S + i4) : run * 0.0f;
    }
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      int b = b1 - e;
      if (b < 0) break;
      *(f32x4*)(g + (size_t)b * S + i4) = run;           // Ghat_b
      const float f = fast_exp2(rx[b] - rx[b + 1]);       // 0 for b = 0 (Rex_0 = -inf)
      run = x[e] + run * f;                               // Ghat_{b-1}
    }
  }
}

// ---------------------------------------------------------------------------
// key side, per chunk b and token j (frame of the boundary gradient: Rex_{b+1}):
//   dchi_j = 2^(R_j - Rex_{b+1}) (Ghat_b v_j + ghat_b) + dchi_intra_j
//   dv_j   = 2^(R_j - Rex_{b+1}) Ghat_b^T chi_j + dv_intra_j
//   dlambda = dchi (*) chi;  dk_j = Omega^T dlambda_j - (sum_p dlambda_jp) k_j
// Four waves per chunk, two chunks per workgroup.  Phase 1: wave w forms
// X = Ghat V^T, dchi and dlambda for feature tiles w, w+4, ... (registers <->
// feature, lanes <-> token) and leaves dlambda and eps chi in LDS; phase 2:
// wave w contracts them over the features for the dk / dv column tiles w, w+4, ...
// ---------------------------------------------------------------------------
template <typename T, int D, int DV, int M>
struct KCfg {
  static constexpr int PAD = MF<T>::PAD;
  static constexpr int TP = tr_pad<T, D>();
  static constexpr int CPB = 2;                       // chunks per workgroup
  static constexpr int WPC = 4;                       // waves per chunk
  static constexpr int ES = sizeof(T);
  static constexpr int a16(int x) { return (x + 15) & ~15; }
  static constexpr int oOm = 0;                                        // Omega*log2 e [p][D]
  static constexpr int oDL = oOm + a16(M * (D + TP) * ES);             // dlambda [c][j][p]
  static constexpr int oCE = oDL + a16(CPB * 32 * (M + PAD) * ES);     // eps chi  [c][j][p]
  static constexpr int oSk = oCE + a16(CPB * 32 * (M + PAD) * ES);     // sum_p dlambda partials
  static constexpr int BYTES = oSk + a16(CPB * WPC * 32 * 4);
};

// A-operand fragment of Ghat rows (float) at k0 in the operand type, hi + lo
template <typename T>
LS_DEV void ghat_frag(const float* row, int k0, typename MF<T>::frag& hi, typename MF<T>::frag& lo) {
  if constexpr (sizeof(T) == 2) {
    const f32x4 x0 = *(const f32x4*)(row + k0), x1 = *(const f32x4*)(row + k0 + 4);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = e < 4 ? x0[e] : x1[e - 4];
      hi[e] = (bf16)x;
      lo[e] = (bf16)(x - (float)hi[e]);
    }
  } else {
    hi = row[k0];
    lo = 0.0f;
  }
}

template <typename T, int D, int DV, int M>
__global__ __launch_bounds__(512) void k_bwd_keys(BwdArgs a, int nfb) {
  using F = MF<T>;
  using C = KCfg<T, D, DV, M>;
  constexpr int PAD = C::PAD, TP = C::TP, WPC = C::WPC;
  constexpr int S = M * DV + M;
  static_assert(C::BYTES <= 160 * 1024, "keys LDS budget");
  __shared__ __align__(16) char smem[C::BYTES];
  T* sOm = (T*)(smem + C::oOm);
  const int tid = threadIdx.x, l = tid & 63, col = l & 31, h = l >> 5, wv = uniform(tid >> 6);
  const int cw = wv / WPC, w = wv % WPC;              // chunk slot, wave within the chunk
  T* sDL = (T*)(smem + C::oDL) + cw * 32 * (M + PAD);
  T* sCE = (T*)(smem + C::oCE) + cw * 32 * (M + PAD);
  float* sSk = (float*)(smem + C::oSk) + cw * WPC * 32;
  const int bh = blockIdx.y, hh = bh % a.H, n = a.n, nch = a.nch;
  const int cb = blockIdx.x * C::CPB + cw;
  const T* omq_h = (const T*)a.omq + (size_t)hh * M * D;
  {
    StageRows<T, M, D, 64 * C::CPB * WPC> so;
    so.load(omq_h, D, 0, 0, M, tid);
    so.store(sOm, D + TP, 0, 0, M, tid);
  }
  const bool active = cb < nch;                       // wave-uniform
  const int cbx = active ? cb : nch - 1;
  const int s0 = cbx * 32;
  const size_t seq = (size_t)bh * n;
  const T* ks = (const T*)a.k + seq * D;
  const T* vs = (const T*)a.v + seq * DV;
  const float* rx = a.rex + (size_t)bh * (nch + 1);
  const float* G = a.gst + ((size_t)bh * nch + cbx) * S;    // Ghat_b [p][d], ghat [p]
  const bool has_after = cbx < nch - 1;
  const int j = s0 + col;
  const bool vt = active && j < n;
  const float eps_j = (vt && has_after) ? fast_exp2(a.rj[seq + j] - rx[cbx + 1]) : 0.0f;

  // ---- phase 1: per feature tile ----
  float sk = 0.0f;
  for (int pt = w; pt < M / 32; pt += WPC) {
    f32x16 X = zero16();
    if (has_after) {
      const float* grow = G + (size_t)(pt * 32 + col) * DV;
#pragma unroll
      for (int s = 0; s < DV / F::KS; ++s) {
        const int k0 = s * F::KS + h * F::KPL;
        typename F::frag hi, lo;
        ghat_frag<T>(grow, k0, hi, lo);
        const typename F::frag vf = vt ? F::ld(vs + (size_t)j * DV, k0) : F::zero();
        X = F::mma(hi, vf, X);
        if constexpr (sizeof(T) == 2) X = F::mma(lo, vf, X);
      }
    }
    // registers <-> p = pt*32 + crow(v, h) (four contiguous per group g), lanes <-> token j
    const T* chirow = (const T*)a.chi + (seq + (vt ? j : s0)) * M;
    const float* dcrow = a.dchi + (seq + (vt ? j : s0)) * M;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int p0 = pt * 32 + 8 * g + 4 * h;
      float ch[4];
      ld4f<T>(chirow + F::sigma(p0), ch);
      const f32x4 di = *(const f32x4*)(dcrow + p0);
      const f32x4 gh = has_after ? *(const f32x4*)(G + (size_t)M * DV + p0) : f32x4{0.f, 0.f, 0.f, 0.f};
      T dl4[4], ce4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float c = vt ? ch[e] : 0.0f;
        const float dc = vt ? eps_j * (X[4 * g + e] + gh[e]) + di[e] : 0.0f;
        dl4[e] = (T)(dc * c * kLn2);                  // paired with Omega * log2(e)
        sk += tof(dl4[e]) * kLog2e;                   // the rounded value the product uses
        ce4[e] = (T)(c * eps_j);
      }
      // natural feature order in LDS (the phase-2 operands read rows j, k = p)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sDL[col * (M + PAD) + p0 + e] = dl4[e];
        sCE[col * (M + PAD) + p0 + e] = ce4[e];
      }
    }
  }
  sk = half_swap_add(sk);
  if (h == 0) sSk[w * 32 + col] = sk;
  __syncthreads();

  // ---- phase 2a: dk column tiles (regs <-> token, lanes <-> D) ----
  for (int Dt = w; Dt < D / 32; Dt += WPC) {
    f32x16 dk = zero16();
#pragma unroll 2
    for (int s = 0; s < M / F::KS; ++s) {
      const int k0 = s * F::KS + h * F::KPL;
      dk = F::mma(F::ld(sDL + col * (M + PAD), k0), F::tld_nat(sOm, D + TP, s * F::KS, Dt * 32), dk);
    }
    if (active) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int jr = crow(v, h), jj = s0 + jr;
        if (jj >= n) continue;
        float skj = 0.0f;
#pragma unroll
        for (int ww = 0; ww < WPC; ++ww) skj += sSk[ww * 32 + jr];
        const int d = Dt * 32 + col;
        ((T*)a.dk)[(seq + jj) * D + d] = (T)(dk[v] - skj * tof(ks[(size_t)jj * D + d]));
      }
    }
  }
  // ---- phase 2b: dv column tiles (regs <-> token, lanes <-> d) ----
  for (int dt = w; dt < DV / 32; dt += WPC) {
    f32x16 dv = zero16();
    if (has_after) {
#pragma unroll 2
      for (int s = 0; s < M / F::KS; ++s) {
        const int k0 = s * F::KS + h * F::KPL;
        // B operand: Ghat rows k0 .. k0 + KPL - 1 (natural k), column dt*32 + col
        typename F::frag hi, lo;
        if constexpr (sizeof(T) == 2) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float x = G[(size_t)(k0 + e) * DV + dt * 32 + col];
            hi[e] = (bf16)x;
            lo[e] = (bf16)(x - (float)hi[e]);
          }
        } else {
          hi = G[(size_t)k0 * DV + dt * 32 + col];
          lo = 0.0f;
        }
        const typename F::frag cf = F::ld(sCE + col * (M + PAD), k0);
        dv = F::mma(cf, hi, dv);
        if constexpr (sizeof(T) == 2) dv = F::mma(cf, lo, dv);
      }
    }
    if (active) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int jj = s0 + crow(v, h);
        if (jj >= n) continue;
        const int d = dt * 32 + col;
        float x = dv[v];
        for (int b = 0; b < nfb; ++b) x += a.dvin[(((size_t)b * a.BH + bh) * n + jj) * DV + d];
        ((T*)a.dv)[(seq + jj) * DV + d] = (T)x;
      }
    }
  }
}

// float32 accumulators (summed over feature blocks) -> output dtype
template <typename T>
__global__ __launch_bounds__(256) void k_bwd_final(const float* __restrict__ src, T* __restrict__ dst,
                                                   size_t count, int nfb) {
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= count) return;
  float x = 0.0f;
  for (int b = 0; b < nfb; ++b) x += src[(size_t)b * count + i];
  dst[i] = (T)x;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
static int launch_err(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("backward %s launch failed: %s", what, hipGetErrorString(e));
    return -4;
  }
  return 0;
}

template <typename T, int D, int DV, int M, int NA>
static int run_bwd(const Shape& s, BwdArgs a, hipStream_t st) {
  using A = AsCfg<T, D, DV, M, NA>;
  constexpr int NFB = A::NFB;
  constexpr int NS = NA + 1;
  const int BH = (int)s.BH();
  const int nch = (int)s.nch();
  const size_t rows = (size_t)BH * s.n;
  {
    ProfScope ps("bwd_prep", st);
    constexpr int RPB = 256 / (DV / (16 / (int)sizeof(T)));     // rows per block of k_bwd_rowprep
    k_bwd_rowprep<T, DV><<<(unsigned)((rows + RPB - 1) / RPB), 256, 0, st>>>(a);
  }
  if (int rc = launch_err("prep")) return rc;
  { ProfScope ps("bwd_du", st);
  k_bwd_du<T, D, DV, M, NA><<<dim3(nch, BH, NFB), 64 * A::NW, 0, st>>>(a);
  }
  if (int rc = launch_err("du")) return rc;
  { ProfScope ps("bwd_dqdr", st);
  k_bwd_dqdr<T, D, DV, M, NA><<<dim3(nch, BH, NFB), 64 * A::NW, 0, st>>>(a);
  }
  if (int rc = launch_err("dqdr")) return rc;
  { ProfScope ps("bwd_state", st);
  k_bwd_state<T, D, DV, M, NA><<<dim3(nch, BH, NFB), 64 * StCfg<T, D, DV, M, NA>::NW, 0, st>>>(a);
  }
  if (int rc = launch_err("state")) return rc;
  constexpr int S = M * DV + M;
  { ProfScope ps("bwd_revscan", st);
  k_bwd_revscan<S><<<dim3((S / 4 + 255) / 256, BH), 256, 0, st>>>(a);
  }
  { ProfScope ps("bwd_keys", st);
  k_bwd_keys<T, D, DV, M><<<dim3((nch + KCfg<T, D, DV, M>::CPB - 1) / KCfg<T, D, DV, M>::CPB, BH), 64 * KCfg<T, D, DV, M>::CPB * KCfg<T, D, DV, M>::WPC, 0, st>>>(a, NFB);
  }
  if (int rc = launch_err("keys")) return rc;
  ProfScope psf("bwd_final", st);
  if constexpr (NFB > 1) {
    k_bwd_final<T><<<(unsigned)((rows * DV + 255) / 256), 256, 0, st>>>(a.du32, (T*)a.du, rows * DV, NFB);
    k_bwd_final<T><<<(unsigned)((rows * D + 255) / 256), 256, 0, st>>>(a.dr32, (T*)a.dr, rows * D, NFB);
  }
  k_bwd_final_dq<T><<<(unsigned)((rows * D / 4 + 255) / 256), 256, 0, st>>>(a.dq32, (T*)a.dq, BH, (int)s.n, D, NFB, NS,
                                                                            s.w);
  return launch_err("final");
}

#define LS_BWD_CASES(X)   \
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

int launch_backward(const Shape& s, const void* q, const void* k, const void* v, const void* r,
                    const void* u, const float* omega, const void* out, const float* stats,
                    const void* dout, void* dq, void* dk, void* dv, void* dr, void* du,
                    const Workspace& ws, hipStream_t st, bool reuse_states) {
  // the forward's prefix states (boundary states and frames): recomputed,
  // unless the caller's workspace still holds them from the forward
  if (!reuse_states) {
    int rc = launch_forward(s, q, k, v, r, u, omega, nullptr, nullptr, nullptr, nullptr, nullptr, ws, st);
    if (rc) return rc;
  }
  BwdArgs a;
  a.q = q; a.k = k; a.v = v; a.r = r; a.u = u; a.omega = omega; a.out = out; a.stats = stats;
  a.dout = dout; a.dq = dq; a.dk = dk; a.dv = dv; a.dr = dr; a.du = du;
  a.omq = ws.omq; a.omk = ws.omk; a.omh = ws.omh; a.states = ws.states; a.states16 = ws.states16; a.rex = ws.rex;
  a.gst = ws.gstates; a.dchi = ws.dchi; a.dvin = ws.dvin; a.du32 = ws.du32; a.dr32 = ws.dr32;
  a.dq32 = ws.dq32; a.rowstat = ws.rowstat; a.chi = ws.chi; a.rj = ws.rj;
  a.H = (int)s.H; a.n = (int)s.n; a.w = s.w; a.nch = (int)s.nch(); a.BH = (int)s.BH();
  a.eps = s.eps;
  const int NA = (s.w + 31) / 32;
#define X(T, D_, DV_, M_)                                                            \
  if (s.dtype == (sizeof(T) == 2 ? 1 : 0) && s.D == D_ && s.Dv == DV_ && s.m == M_) { \
    if (NA == 1) return run_bwd<T, D_, DV_, M_, 1>(s, a, st);                        \
    if (NA == 2) return run_bwd<T, D_, DV_, M_, 2>(s, a, st);                        \
    if constexpr (wide_window_ok(sizeof(T) == 2 ? 1 : 0, D_, M_, 3)) {                \
      if (NA == 3) return run_bwd<T, D_, DV_, M_, 3>(s, a, st);                      \
    }                                                                                \
    if constexpr (wide_window_ok(sizeof(T) == 2 ? 1 : 0, D_, M_, 4)) {                \
      if (NA == 4) return run_bwd<T, D_, DV_, M_, 4>(s, a, st);                      \
    }                                                                                \
  }
  LS_BWD_CASES(X)
#undef X
  set_error("backward: unsupported shape (dtype=%d D=%d Dv=%d m=%d)", s.dtype, s.D, s.Dv, s.m);
  return -2;
}

}  // namespace linsimp
