// Key-side log-features shared by the forward kernels (chunk states, key features).
#pragma once
#include "common.h"

namespace linsimp {

// ---------------------------------------------------------------------------
// The key-side bank copy (Omega log2 e, M x D per head, bf16 hi then lo halves)
// is kept in matrix-core fragment order: for feature tile pt, k-step s and lane
// (h, col), the KPL elements of row 32 pt + col, columns s KS + h KPL onwards,
// are contiguous, so one fragment load of a wave reads 64 KPL contiguous
// elements (a row-major bank spreads it over 32 rows).
// ---------------------------------------------------------------------------
template <typename T, int D>
LS_DEV size_t bank_frag(int pt, int s, int lane) {
  using F = MF<T>;
  return ((size_t)(pt * (D / F::KS) + s) * 64 + lane) * F::KPL;
}

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
      typename F::frag of = *(const typename F::frag*)(omk_h + bank_frag<T, D>(pt, s, l));
      acc[pt] = TOKEN_COLS ? F::mma(of, kf, acc[pt]) : F::mma(kf, of, acc[pt]);
      if constexpr (sizeof(T) == 2) {
        typename F::frag ol = *(const typename F::frag*)(omk_h + (size_t)M * D + bank_frag<T, D>(pt, s, l));
        acc[pt] = TOKEN_COLS ? F::mma(ol, kf, acc[pt]) : F::mma(kf, ol, acc[pt]);
      }
    }
  }
  nk = half_swap_add(nk);
}


}  // namespace linsimp
