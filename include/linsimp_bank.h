/*
 * linsimp_bank.h -- C ABI of the orthogonal random-feature bank sampler of
 * the LinSimp paper (App. B.1, "Orthogonal Gaussian marginals").
 *
 * For every head h and block b = 0 .. nb-1 (nb = ceil(m / D)):
 *   1. G = QR, G the block's D x D draw of iid N(0, 1) entries;
 *   2. with sign_correct, column a of Q is multiplied by sign(R_aa) (the
 *      step that makes Q Haar-distributed);
 *   3. row b*D + a of the bank is column a of Q times the radius r_a (a chi_D
 *      draw), so every row has the N(0, I_D) marginal of Lemma 1;
 *   4. blocks are stacked and the bank is cut to m rows.
 * The random draws are inputs: the caller supplies G and the radii (e.g. the
 * norms of D-dimensional standard normal vectors, which are chi_D).  The
 * factorisation runs in float64 (Householder, R_aa = -sign(x_a)|x|); the bank
 * is written as float32, the layout every linsimp entry point takes.
 *
 * Conventions as in linsimp.h (device pointers, 16-byte aligned, no
 * allocation, enqueue-only, negative linsimp_status on error).
 */
#ifndef LINSIMP_BANK_H
#define LINSIMP_BANK_H

#include "linsimp.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Orthogonal feature bank for H heads.
 *   gauss : [H, nb, D, D] float32, block b of head h row-major (G[i][j])
 *   radii : [H, nb, D] float32
 *   omega : [H, m, D] float32, written
 *   sign_correct : 1 for the paper's sampler; 0 keeps the raw Householder
 *                  factor (the variant App. B.1 reports as biased)
 * D in {32, 64, 128}; H >= 1; m >= 1.  Uses no workspace. */
int linsimp_feature_bank(int32_t H, int32_t m, int32_t D, const float* gauss, const float* radii,
                         float* omega, int32_t sign_correct, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LINSIMP_BANK_H */
