// The steps either side of the LinSimp core that make up one attention head
// (paper Sec. 3.1 and eq:gated-output):
//
//   before the core:  q' = tau_h * q / |q|,  k' = k / |k|,  r' = r / |r|
//   after the core:   y = g (*) o~ / sqrt(mean(o~^2) + rms_eps)
//                     g = sigmoid(gamma_h)  (one gate per head)  or
//                     g = sigmoid(l_i)      (channel-wise gate, logits l_i given)
//
// plus their exact backward.  |x| is floored at norm_eps (x / norm_eps below
// the floor).  Every kernel is a streaming row pass (HBM-bound): 16 lanes per
// row (four rows per wave, each lane one contiguous 16-byte piece of a bf16
// row of 128), float32 arithmetic, row sums by DPP within the 16-lane row.
// Per-head sums (dtau, dgamma) go through per-row partials and a fixed-order
// reduction (deterministic).
#include <hip/hip_runtime.h>

#include "common.h"
#include "linsimp_internal.h"
#include "prof.h"

namespace linsimp {

namespace {

constexpr int kRowsPerBlock = 16;   // 16 lanes per row, four rows per wave, four waves

LS_DEV float sigmoidf(float x) { return 1.0f / (1.0f + expf(-x)); }

// sum over the 16 lanes of a DPP row (every lane gets the sum)
LS_DEV float row16_sum(float x) {
  x += dpp<0xB1>(x);      // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);      // quad_perm [2,3,0,1]
  x += dpp<0x124>(x);     // row_ror:4
  x += dpp<0x128>(x);     // row_ror:8
  return x;
}

// the lane's contiguous piece of a row of width W: elements [sub E, sub E + E)
template <int W> struct RowVec {
  static constexpr int E = W / 16;
  float x[E];
  template <typename T> LS_DEV void load(const T* row, int sub) {
    typedef T V __attribute__((ext_vector_type(E)));
    const V v = *(const V*)(row + sub * E);
#pragma unroll
    for (int j = 0; j < E; ++j) x[j] = tof(v[j]);
  }
  template <typename T> LS_DEV void store(T* row, int sub) const {
    typedef T V __attribute__((ext_vector_type(E)));
    V v;
#pragma unroll
    for (int j = 0; j < E; ++j) v[j] = fromf<T>(x[j]);
    *(V*)(row + sub * E) = v;
  }
  LS_DEV float dot(const RowVec& o) const {
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < E; ++j) s += x[j] * o.x[j];
    return row16_sum(s);
  }
};

// row handled by this lane's 16-lane group, and the lane's index in it
#define LS_HEAD_ROW                                                                  \
  const int sub = threadIdx.x & 15;                                                   \
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 4);       \
  if (row >= rows) return;

// ---------------------------------------------------------------------------
// forward: L2 normalisation of q, k, r (q also times tau_h)
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(16 * kRowsPerBlock) void k_head_prenorm(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ r,
    const float* __restrict__ tau, T* __restrict__ qn, T* __restrict__ kn, T* __restrict__ rn,
    int64_t rows, int64_t n, int H, float norm_eps) {
  LS_HEAD_ROW
  const int hh = (int)((row / n) % H);
  const size_t off = (size_t)row * D;
  const T* src[3] = {q + off, k + off, r + off};
  T* dst[3] = {qn + off, kn + off, rn + off};
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    RowVec<D> x;
    x.load(src[s], sub);
    const float nrm = fmaxf(sqrtf(x.dot(x)), norm_eps);
    const float scale = (s == 0 ? tau[hh] : 1.0f) / nrm;
#pragma unroll
    for (int j = 0; j < RowVec<D>::E; ++j) x.x[j] *= scale;
    x.store(dst[s], sub);
  }
}

// ---------------------------------------------------------------------------
// forward: gated RMSNorm of the core output; keeps rho = 1/sqrt(ms + eps)
// ---------------------------------------------------------------------------
template <typename T, int DV, bool CHANNEL>
__global__ __launch_bounds__(16 * kRowsPerBlock) void k_head_gate(
    const T* __restrict__ ot, const void* __restrict__ gate, T* __restrict__ y,
    float* __restrict__ rho_out, int64_t rows, int64_t n, int H, float rms_eps) {
  LS_HEAD_ROW
  const size_t off = (size_t)row * DV;
  RowVec<DV> o;
  o.load(ot + off, sub);
  const float rho = 1.0f / sqrtf(o.dot(o) / (float)DV + rms_eps);
  RowVec<DV> g;
  if constexpr (CHANNEL) {
    g.load((const T*)gate + off, sub);
#pragma unroll
    for (int j = 0; j < RowVec<DV>::E; ++j) g.x[j] = sigmoidf(g.x[j]);
  } else {
    const float gh = sigmoidf(((const float*)gate)[(row / n) % H]);
#pragma unroll
    for (int j = 0; j < RowVec<DV>::E; ++j) g.x[j] = gh;
  }
#pragma unroll
  for (int j = 0; j < RowVec<DV>::E; ++j) o.x[j] *= rho * g.x[j];
  o.store(y + off, sub);
  if (sub == 0) rho_out[row] = rho;
}

// ---------------------------------------------------------------------------
// backward: gated RMSNorm.  Writes d o~ (the core's upstream gradient) and
// either d logits (channel gate) or the row's share of d gamma.
// ---------------------------------------------------------------------------
template <typename T, int DV, bool CHANNEL>
__global__ __launch_bounds__(16 * kRowsPerBlock) void k_head_gate_bwd(
    const T* __restrict__ ot, const float* __restrict__ rho_in, const void* __restrict__ gate,
    const T* __restrict__ dy, T* __restrict__ dot_out, void* __restrict__ dgate,
    float* __restrict__ part, int64_t rows, int64_t n, int H) {
  LS_HEAD_ROW
  const size_t off = (size_t)row * DV;
  const float rho = rho_in[row];
  RowVec<DV> oh, g, d;
  oh.load(ot + off, sub);
#pragma unroll
  for (int j = 0; j < RowVec<DV>::E; ++j) oh.x[j] *= rho;
  d.load(dy + off, sub);
  if constexpr (CHANNEL) {
    g.load((const T*)gate + off, sub);
#pragma unroll
    for (int j = 0; j < RowVec<DV>::E; ++j) g.x[j] = sigmoidf(g.x[j]);
  } else {
    const float gh = sigmoidf(((const float*)gate)[(row / n) % H]);
#pragma unroll
    for (int j = 0; j < RowVec<DV>::E; ++j) g.x[j] = gh;
  }
  // gate derivative dy * o_hat * g (1 - g)
  RowVec<DV> dl;
  float dls = 0.0f;
#pragma unroll
  for (int j = 0; j < RowVec<DV>::E; ++j) {
    dl.x[j] = d.x[j] * oh.x[j] * g.x[j] * (1.0f - g.x[j]);
    dls += dl.x[j];
  }
  if constexpr (CHANNEL) {
    dl.store((T*)dgate + off, sub);
  } else {
    dls = row16_sum(dls);
    if (sub == 0) part[row] = dls;
  }
  // RMSNorm: d o~ = rho (d o_hat - o_hat (d o_hat . o_hat) / DV),  d o_hat = g dy
#pragma unroll
  for (int j = 0; j < RowVec<DV>::E; ++j) d.x[j] *= g.x[j];
  const float s = d.dot(oh) / (float)DV;
#pragma unroll
  for (int j = 0; j < RowVec<DV>::E; ++j) d.x[j] = rho * (d.x[j] - oh.x[j] * s);
  d.store(dot_out + off, sub);
}

// ---------------------------------------------------------------------------
// backward: L2 normalisation and temperature.  dx (in: the core's gradient
// with respect to the normalised input; out: the gradient with respect to x)
// may alias; the row's share of dtau goes to part.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(16 * kRowsPerBlock) void k_head_prenorm_bwd(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ r,
    const float* __restrict__ tau, T* dq, T* dk, T* dr, float* __restrict__ part, int64_t rows,
    int64_t n, int H, float norm_eps) {
  LS_HEAD_ROW
  const int hh = (int)((row / n) % H);
  const size_t off = (size_t)row * D;
  const T* src[3] = {q + off, k + off, r + off};
  T* grad[3] = {dq + off, dk + off, dr + off};
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    RowVec<D> x, g;
    x.load(src[s], sub);
    g.load(grad[s], sub);
    const float nr = sqrtf(x.dot(x));
    const float inv = 1.0f / fmaxf(nr, norm_eps);
#pragma unroll
    for (int j = 0; j < RowVec<D>::E; ++j) x.x[j] *= inv;          // x_hat
    if (s == 0) {
      const float dt = x.dot(g);                                    // x_hat . d(core q)
      if (sub == 0) part[row] = dt;
      const float t = tau[hh];
#pragma unroll
      for (int j = 0; j < RowVec<D>::E; ++j) g.x[j] *= t;          // d x_hat
    }
    if (nr > norm_eps) {
      const float p = x.dot(g);
#pragma unroll
      for (int j = 0; j < RowVec<D>::E; ++j) g.x[j] = (g.x[j] - x.x[j] * p) * inv;
    } else {
#pragma unroll
      for (int j = 0; j < RowVec<D>::E; ++j) g.x[j] *= inv;
    }
    g.store(grad[s], sub);
  }
}

// per-head sums of per-row partials: out[h] = sum over b, i of part[(b H + h) n + i]
__global__ __launch_bounds__(256) void k_head_reduce(const float* __restrict__ part, float* __restrict__ out,
                                                     int64_t B, int64_t n, int H) {
  __shared__ float red[256];
  const int hh = blockIdx.x, t = threadIdx.x;
  float s = 0.0f;
  for (int64_t b = 0; b < B; ++b) {
    const float* p = part + ((size_t)b * H + hh) * n;
    for (int64_t i = t; i < n; i += 256) s += p[i];
  }
  red[t] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] += red[t + o];
    __syncthreads();
  }
  if (t == 0) out[hh] = red[0];
}

int launch_err(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("head %s launch failed: %s", what, hipGetErrorString(e));
    return -4;
  }
  return 0;
}

unsigned row_blocks(int64_t rows) { return (unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock); }

template <typename T, int D>
int prenorm_t(const Shape& s, const void* q, const void* k, const void* r, const float* tau, void* qn,
              void* kn, void* rn, float norm_eps, hipStream_t st) {
  const int64_t rows = s.BH() * s.n;
  ProfScope ps("head_prenorm", st);
  k_head_prenorm<T, D><<<row_blocks(rows), 16 * kRowsPerBlock, 0, st>>>(
      (const T*)q, (const T*)k, (const T*)r, tau, (T*)qn, (T*)kn, (T*)rn, rows, s.n, (int)s.H, norm_eps);
  return launch_err("prenorm");
}

template <typename T, int DV>
int gate_t(const Shape& s, const void* ot, const void* gate, bool channel, void* y, float* rho,
           float rms_eps, hipStream_t st) {
  const int64_t rows = s.BH() * s.n;
  ProfScope ps("head_gate", st);
  if (channel)
    k_head_gate<T, DV, true><<<row_blocks(rows), 16 * kRowsPerBlock, 0, st>>>(
        (const T*)ot, gate, (T*)y, rho, rows, s.n, (int)s.H, rms_eps);
  else
    k_head_gate<T, DV, false><<<row_blocks(rows), 16 * kRowsPerBlock, 0, st>>>(
        (const T*)ot, gate, (T*)y, rho, rows, s.n, (int)s.H, rms_eps);
  return launch_err("gate");
}

template <typename T, int DV>
int gate_bwd_t(const Shape& s, const void* ot, const float* rho, const void* gate, bool channel,
               const void* dy, void* dot, void* dgate, float* part, hipStream_t st) {
  const int64_t rows = s.BH() * s.n;
  ProfScope ps("head_gate_bwd", st);
  if (channel)
    k_head_gate_bwd<T, DV, true><<<row_blocks(rows), 16 * kRowsPerBlock, 0, st>>>(
        (const T*)ot, rho, gate, (const T*)dy, (T*)dot, dgate, part, rows, s.n, (int)s.H);
  else
    k_head_gate_bwd<T, DV, false><<<row_blocks(rows), 16 * kRowsPerBlock, 0, st>>>(
        (const T*)ot, rho, gate, (const T*)dy, (T*)dot, dgate, part, rows, s.n, (int)s.H);
  return launch_err("gate_bwd");
}

template <typename T, int D>
int prenorm_bwd_t(const Shape& s, const void* q, const void* k, const void* r, const float* tau,
                  void* dq, void* dk, void* dr, float* part, float norm_eps, hipStream_t st) {
  const int64_t rows = s.BH() * s.n;
  ProfScope ps("head_prenorm_bwd", st);
  k_head_prenorm_bwd<T, D><<<row_blocks(rows), 16 * kRowsPerBlock, 0, st>>>(
      (const T*)q, (const T*)k, (const T*)r, tau, (T*)dq, (T*)dk, (T*)dr, part, rows, s.n, (int)s.H,
      norm_eps);
  return launch_err("prenorm_bwd");
}

template <typename T>
int prenorm_d(const Shape& s, const void* q, const void* k, const void* r, const float* tau, void* qn,
              void* kn, void* rn, float norm_eps, hipStream_t st) {
  switch (s.D) {
    case 32: return prenorm_t<T, 32>(s, q, k, r, tau, qn, kn, rn, norm_eps, st);
    case 64: return prenorm_t<T, 64>(s, q, k, r, tau, qn, kn, rn, norm_eps, st);
    case 128: return prenorm_t<T, 128>(s, q, k, r, tau, qn, kn, rn, norm_eps, st);
  }
  set_error("head: unsupported D=%d", s.D);
  return -2;
}

template <typename T>
int gate_d(const Shape& s, const void* ot, const void* gate, bool channel, void* y, float* rho,
           float rms_eps, hipStream_t st) {
  switch (s.Dv) {
    case 32: return gate_t<T, 32>(s, ot, gate, channel, y, rho, rms_eps, st);
    case 64: return gate_t<T, 64>(s, ot, gate, channel, y, rho, rms_eps, st);
    case 128: return gate_t<T, 128>(s, ot, gate, channel, y, rho, rms_eps, st);
  }
  set_error("head: unsupported Dv=%d", s.Dv);
  return -2;
}

template <typename T>
int gate_bwd_d(const Shape& s, const void* ot, const float* rho, const void* gate, bool channel,
               const void* dy, void* dot, void* dgate, float* part, hipStream_t st) {
  switch (s.Dv) {
    case 32: return gate_bwd_t<T, 32>(s, ot, rho, gate, channel, dy, dot, dgate, part, st);
    case 64: return gate_bwd_t<T, 64>(s, ot, rho, gate, channel, dy, dot, dgate, part, st);
    case 128: return gate_bwd_t<T, 128>(s, ot, rho, gate, channel, dy, dot, dgate, part, st);
  }
  set_error("head: unsupported Dv=%d", s.Dv);
  return -2;
}

template <typename T>
int prenorm_bwd_d(const Shape& s, const void* q, const void* k, const void* r, const float* tau,
                  void* dq, void* dk, void* dr, float* part, float norm_eps, hipStream_t st) {
  switch (s.D) {
    case 32: return prenorm_bwd_t<T, 32>(s, q, k, r, tau, dq, dk, dr, part, norm_eps, st);
    case 64: return prenorm_bwd_t<T, 64>(s, q, k, r, tau, dq, dk, dr, part, norm_eps, st);
    case 128: return prenorm_bwd_t<T, 128>(s, q, k, r, tau, dq, dk, dr, part, norm_eps, st);
  }
  set_error("head: unsupported D=%d", s.D);
  return -2;
}

}  // namespace

int launch_head_prenorm(const Shape& s, const void* q, const void* k, const void* r, const float* tau,
                        void* qn, void* kn, void* rn, float norm_eps, hipStream_t st) {
  return s.dtype == 1 ? prenorm_d<bf16>(s, q, k, r, tau, qn, kn, rn, norm_eps, st)
                      : prenorm_d<float>(s, q, k, r, tau, qn, kn, rn, norm_eps, st);
}

int launch_head_gate(const Shape& s, const void* ot, const void* gate, bool channel, void* y,
                     float* rho, float rms_eps, hipStream_t st) {
  return s.dtype == 1 ? gate_d<bf16>(s, ot, gate, channel, y, rho, rms_eps, st)
                      : gate_d<float>(s, ot, gate, channel, y, rho, rms_eps, st);
}

int launch_head_gate_bwd(const Shape& s, const void* ot, const float* rho, const void* gate,
                         bool channel, const void* dy, void* dot, void* dgate, float* part,
                         hipStream_t st) {
  return s.dtype == 1 ? gate_bwd_d<bf16>(s, ot, rho, gate, channel, dy, dot, dgate, part, st)
                      : gate_bwd_d<float>(s, ot, rho, gate, channel, dy, dot, dgate, part, st);
}

int launch_head_prenorm_bwd(const Shape& s, const void* q, const void* k, const void* r,
                            const float* tau, void* dq, void* dk, void* dr, float* part,
                            float norm_eps, hipStream_t st) {
  return s.dtype == 1 ? prenorm_bwd_d<bf16>(s, q, k, r, tau, dq, dk, dr, part, norm_eps, st)
                      : prenorm_bwd_d<float>(s, q, k, r, tau, dq, dk, dr, part, norm_eps, st);
}

int launch_head_reduce(const Shape& s, const float* part, float* out, hipStream_t st) {
  ProfScope ps("head_reduce", st);
  k_head_reduce<<<(unsigned)s.H, 256, 0, st>>>(part, out, s.B, s.n, (int)s.H);
  return launch_err("reduce");
}

}  // namespace linsimp
