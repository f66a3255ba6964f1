// Orthogonal random-feature bank (paper App. B.1) from given Gaussian draws.
//
// For each head h and block b (nb = ceil(m / D) blocks per head):
//   G = QR                      Householder factorisation of the D x D draw
//   Q <- Q diag(sign(R_aa))     when sign correction is on (Haar factor)
//   Omega[h][b D + a] = radius[h][b][a] * (column a of Q), a = 0 .. D-1
// truncated to m rows.  One workgroup per (block, head); the factorisation
// runs in float64 in LDS (the matrix is stored by columns), the output is
// float32.  The Householder vectors follow the usual convention
// R_kk = -sign(x_k) |x| (sign(0) = +1), v_k = 1, so with the correction off
// the factor is the one LAPACK-style QR returns.
//
// Q is formed in place by backward accumulation, Q = H_0 (H_1 (... H_{D-1})),
// which only ever touches the trailing block of rows and columns i.. .
#include <hip/hip_runtime.h>

#include "linsimp_internal.h"
#include "prof.h"

namespace linsimp {

namespace {

constexpr int kBankThreads = 256;

__device__ double block_sum(double x, double* red) {
  const int t = threadIdx.x;
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  if ((t & 63) == 0) red[t >> 6] = x;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int w = 0; w < kBankThreads / 64; ++w) s += red[w];
  __syncthreads();
  return s;
}

template <int D>
__global__ __launch_bounds__(kBankThreads) void k_feature_bank(const float* __restrict__ gauss,
                                                                const float* __restrict__ radii,
                                                                float* __restrict__ omega, int m,
                                                                int sign_correct) {
  constexpr int LD = D + 1;                     // column stride (doubles)
  __shared__ double A[D * LD];                  // A[j * LD + i] = entry (i, j)
  __shared__ double tau[D], rdiag[D], w[D], red[kBankThreads / 64];
  const int t = threadIdx.x;
  const int b = blockIdx.x, hh = blockIdx.y, nb = gridDim.x;
  const float* G = gauss + ((size_t)hh * nb + b) * D * D;
  for (int e = t; e < D * D; e += kBankThreads) {
    const int i = e / D, j = e % D;             // G row-major [i][j]
    A[j * LD + i] = (double)G[e];
  }
  __syncthreads();

  // ---- Householder factorisation, column by column ----
  for (int k = 0; k < D; ++k) {
    double* col = A + k * LD;
    double ss = 0.0;
    for (int i = k + 1 + t; i < D; i += kBankThreads) ss += col[i] * col[i];
    const double xn2 = block_sum(ss, red);
    const double alpha = col[k];
    double beta = alpha, tk = 0.0, scale = 0.0;
    if (xn2 > 0.0) {
      const double nrm = sqrt(alpha * alpha + xn2);
      beta = alpha >= 0.0 ? -nrm : nrm;
      tk = (beta - alpha) / beta;
      scale = 1.0 / (alpha - beta);
    }
    __syncthreads();
    if (t == 0) {
      tau[k] = tk;
      rdiag[k] = beta;
      col[k] = 1.0;                              // v_k = 1 while the reflector is applied
    }
    if (xn2 > 0.0)
      for (int i = k + 1 + t; i < D; i += kBankThreads) col[i] *= scale;
    __syncthreads();
    // w_j = v^T A[k:, j] for the trailing columns, then A[k:, j] -= tau v w_j
    if (tk != 0.0) {
      for (int j = k + 1 + t; j < D; j += kBankThreads) {
        const double* cj = A + j * LD;
        double s = 0.0;
        for (int i = k; i < D; ++i) s += col[i] * cj[i];
        w[j] = s;
      }
      __syncthreads();
      const int rows = D - k, cols = D - k - 1;
      for (int e = t; e < rows * cols; e += kBankThreads) {
        const int i = k + e % rows, j = k + 1 + e / rows;
        A[j * LD + i] -= tk * col[i] * w[j];
      }
    }
    __syncthreads();
    if (t == 0) col[k] = beta;                   // R_kk (kept in rdiag too)
    __syncthreads();
  }

  // ---- Q by backward accumulation, in place ----
  for (int k = D - 1; k >= 0; --k) {
    double* col = A + k * LD;
    const double tk = tau[k];
    if (t == 0) col[k] = 1.0;
    __syncthreads();
    if (k < D - 1 && tk != 0.0) {
      for (int j = k + 1 + t; j < D; j += kBankThreads) {
        const double* cj = A + j * LD;
        double s = 0.0;
        for (int i = k; i < D; ++i) s += col[i] * cj[i];
        w[j] = s;
      }
      __syncthreads();
      const int rows = D - k, cols = D - k - 1;
      for (int e = t; e < rows * cols; e += kBankThreads) {
        const int i = k + e % rows, j = k + 1 + e / rows;
        A[j * LD + i] -= tk * col[i] * w[j];
      }
      __syncthreads();
    }
    // column k of Q: e_k - tau v (entries above k are zero)
    for (int i = t; i < D; i += kBankThreads) {
      if (i < k) col[i] = 0.0;
      else if (i == k) col[i] = 1.0 - tk;
      else col[i] = -tk * col[i];
    }
    __syncthreads();
  }

  // ---- sign correction, radii, output rows b*D + a ----
  const float* rad = radii + ((size_t)hh * nb + b) * D;
  for (int e = t; e < D * D; e += kBankThreads) {
    const int a = e / D, i = e % D;
    const int row = b * D + a;
    if (row >= m) continue;
    double s = (double)rad[a];
    if (sign_correct && rdiag[a] < 0.0) s = -s;
    omega[((size_t)hh * m + row) * D + i] = (float)(s * A[a * LD + i]);
  }
}

}  // namespace

int launch_feature_bank(int H, int m, int D, const float* gauss, const float* radii, float* omega,
                        int sign_correct, hipStream_t st) {
  const int nb = (m + D - 1) / D;
  const dim3 grid(nb, H);
  ProfScope ps("feature_bank", st);
  switch (D) {
    case 32: k_feature_bank<32><<<grid, kBankThreads, 0, st>>>(gauss, radii, omega, m, sign_correct); break;
    case 64: k_feature_bank<64><<<grid, kBankThreads, 0, st>>>(gauss, radii, omega, m, sign_correct); break;
    case 128: k_feature_bank<128><<<grid, kBankThreads, 0, st>>>(gauss, radii, omega, m, sign_correct); break;
    default:
      set_error("feature bank: D=%d not in {32, 64, 128}", D);
      return -2;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("feature bank launch failed: %s", hipGetErrorString(e));
    return -4;
  }
  return 0;
}

}  // namespace linsimp
