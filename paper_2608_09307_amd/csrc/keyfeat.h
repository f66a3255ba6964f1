// Key-side feature map shared by the forward, backward and prefill kernels.
#pragma once
#include "common.h"

namespace linsimp {

// ---------------------------------------------------------------------------
// Key log2-features of 32 tokens [tok0, tok0+32) against all M feature rows.
// TOKEN_COLS: lanes <-> token, registers <-> feature p (acc[pt] rows p = 32pt+crow).
// else      : lanes <-> feature p, registers <-> token.
// The |k|^2/2 term is not applied; nk returns |k_tok|^2 for the lane's token.
// ---------------------------------------------------------------------------
template <typename T, int D, int M, bool TOKEN_COLS>
LS_DEV void key_logits(f32x16 (&acc)[M / 32], float& nk, const T* __restrict__ kseq, int tok0, int n,
                       const T* __restrict__ omk_h) {
  using F = MF<T>;
  const int l = lane_id(), col = l & 31, h = l >> 5;
  const int j = tok0 + col;
  const bool vj = j < n;
#pragma unroll
  for (int pt = 0; pt < M / 32; ++pt) acc[pt] = zero16();
  nk = 0.0f;
#pragma unroll 1
  for (int s = 0; s < D / F::KS; ++s) {
    const int k0 = s * F::KS + h * F::KPL;
    typename F::frag kf = vj ? F::ld(kseq + (size_t)j * D, k0) : F::zero();
#pragma unroll
    for (int e = 0; e < F::KPL; ++e) { float x = fel(kf, e); nk += x * x; }
#pragma unroll
    for (int pt = 0; pt < M / 32; ++pt) {
      typename F::frag of = F::ld(omk_h + (size_t)(pt * 32 + col) * D, k0);
      acc[pt] = TOKEN_COLS ? F::mma(of, kf, acc[pt]) : F::mma(kf, of, acc[pt]);
      if constexpr (sizeof(T) == 2) {
        typename F::frag ol = F::ld(omk_h + (size_t)M * D + (size_t)(pt * 32 + col) * D, k0);
        acc[pt] = TOKEN_COLS ? F::mma(ol, kf, acc[pt]) : F::mma(kf, ol, acc[pt]);
      }
    }
  }
  nk = half_swap_add(nk);
}


// Key features of the 32 tokens of one chunk, computed by one wave:
//   R_j = max(Rexb, max_{s0 <= j' <= j} max_p lambda_j'p)   (causal running frame, log2)
//   chi_j = 2^(lambda_j - R_j) / sqrt(M)
// written as sChi[j * chi_ld + sigma(p - p_lo)] for p in [p_lo, p_hi) (type T)
// and sRj[j].  Tokens >= n get 0.
template <typename T, int D, int M>
LS_DEV void chunk_key_features(const T* __restrict__ ks, int s0, int n, const T* __restrict__ omk_h,
                               float Rexb, T* sChi, int chi_ld, float* sRj, int p_lo = 0,
                               int p_hi = M) {
  using F = MF<T>;
  const int l = lane_id(), col = l & 31, h = l >> 5;
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
  R = fmaxf(R, Rexb);
  if (h == 0) sRj[col] = R;
  const float rsm = rsqrtf((float)M);
  T* row = sChi + col * chi_ld;
#pragma unroll
  for (int pt = 0; pt < M / 32; ++pt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      int p = pt * 32 + crow(v, h);
      if (p >= p_lo && p < p_hi) row[F::sigma(p - p_lo)] = (T)(fast_exp2(acc[pt][v] - R) * rsm);
    }
}

}  // namespace linsimp
