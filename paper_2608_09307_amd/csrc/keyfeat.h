// Key-side log-features shared by the forward kernels (chunk states, key features).
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
    typename F::frag kf = F::ld(kseq + (size_t)min(j, n - 1) * D, k0);
    if (!vj) kf = F::zero();
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


}  // namespace linsimp
