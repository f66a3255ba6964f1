// Internal (host + device) declarations shared by the LinSimp HIP sources.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace linsimp {

// Sequence chunk used by every kernel: key chunks for the prefix-state scan and
// the row chunks of the readout share it.
constexpr int kChunk = 32;

struct Shape {
  int64_t B, H, n;
  int D, Dv, m, w;
  int dtype;   // 0 = f32, 1 = bf16
  float eps;
  int64_t BH() const { return B * H; }
  int64_t nch() const { return (n + kChunk - 1) / kChunk; }
  int64_t state_elems() const { return (int64_t)m * Dv + m; }   // M (m x Dv) then a (m)
  size_t esize() const { return dtype == 1 ? 2 : 4; }
};

// Workspace carve shared by forward and backward.
struct Workspace {
  void* omq;        // [H][m][D] operand type: query-side Omega * log2(e)
  void* omk;        // bf16: [H][2][m*D] hi/lo split of Omega*log2(e); f32: [H][m*D]; fragment order
  void* omh;        // [H][m][D] f16 Omega*log2(e): the query-side logits of bf16 inputs
  float* states;    // [BH][nch][m*Dv + m]  chunk contributions, then boundary states (bf16 inputs: a only;
                   //                      the M slot holds the chunk's chi^T and V^T operand fragments)
  void* states16;   // [BH][nch][m*Dv]      bf16 inputs: the boundary states' M, in bf16 (the operand type of
                   //                      every reader); states then keeps the chunk contributions' M
  float* rho;       // [BH][nch]            chunk max of key log2-features
  float* rex;       // [BH][nch + 1]        frame (log2) of each boundary state; [nch] = final
  void* chi;        // [BH][n][m] operand type: key features 2^(lambda_j - R_j)/sqrt(m), p permuted in 16-blocks
  float* rj;        // [BH][n]              running key frame R_j (log2)
  float* part;      // [m/128][BH][n][Dv+2] per-feature-block readout partials (m > 128)
  // backward-only regions (null in forward)
  float* gstates;   // [BH][nch][m*Dv + m]  per-chunk state gradients, then reverse-scanned
  float* dchi;      // [BH][n][m]           intra-chunk key-feature gradient (frame R_j)
  float* dvin;      // [nfb][BH][n][Dv]     intra-chunk value gradient
  float* du32;      // [nfb][BH][n][Dv]     du per feature block (m > 128 only)
  float* dr32;      // [nfb][BH][n][D]      dr per feature block (m > 128 only)
  float* dq32;      // [nfb][ns][BH][n][D]  dq partial of each anchor tile (slot = row chunk - anchor tile)
  float* rowstat;   // [BH][n][2]           per-row 1/(Z+eps) and dZ
};

// Windows wider than 64 (NA = ceil(w / 32) = 3 or 4 anchor tiles per row)
// follow the launch rule w * min(m, 128) <= 8192: m <= 64.  The one exception
// is float32 with D = m = 64 at NA = 4, whose du sweep would need 167 KB of
// LDS for its five staged row chunks.
constexpr bool wide_window_ok(int dtype, int D, int m, int NA) {
  return NA <= 2 || (NA <= 4 && m <= 64 && 32 * NA * m <= 8192 && !(dtype == 0 && D == 64 && m == 64 && NA == 4));
}

// Row-side dq is summed over the anchor tiles a row sees: row i receives from
// tiles floor(i/32) - ns + 1 .. floor(i/32), ns = ceil(w/32) + 1.
inline int bwd_slots(int w) { return (w + kChunk - 1) / kChunk + 1; }
// feature blocks of the backward (128 features each, fewer for m < 128)
inline int bwd_nfb(int m) { return m > 128 ? m / 128 : 1; }

size_t workspace_bytes(const Shape& s, bool backward);
void carve(const Shape& s, void* base, bool backward, Workspace* ws);

// Returns 0 on success, negative linsimp status otherwise (message via set_error).
int launch_forward(const Shape& s, const void* q, const void* k, const void* v, const void* r,
                   const void* u, const float* omega, void* out, float* stats,
                   float* final_M, float* final_a, float* final_rex, const Workspace& ws,
                   hipStream_t st);
bool fwd_combo_supported(int dtype, int D, int Dv, int m);
int launch_ring_fill(const Shape& s, const void* r, const void* u, void* ring_r, void* ring_u,
                     int64_t* pos, hipStream_t st);

int launch_backward(const Shape& s, const void* q, const void* k, const void* v, const void* r,
                    const void* u, const float* omega, const void* out, const float* stats,
                    const void* dout, void* dq, void* dk, void* dv, void* dr, void* du,
                    const Workspace& ws, hipStream_t st, bool reuse_states = false);

int launch_decode(int64_t S, int H, int ntok, int D, int Dv, int m, int w, int dtype, float eps,
                  const void* q, const void* k, const void* v, const void* r, const void* u,
                  const float* omega, float* M, float* a, float* rho, void* ring_r, void* ring_u,
                  int64_t* pos, void* out, hipStream_t st);

// steps of the full head around the core (head.hip)
int launch_head_prenorm(const Shape& s, const void* q, const void* k, const void* r, const float* tau,
                        void* qn, void* kn, void* rn, float norm_eps, hipStream_t st);
int launch_head_gate(const Shape& s, const void* ot, const void* gate, bool channel, void* y,
                     float* rho, float rms_eps, hipStream_t st);
int launch_head_gate_bwd(const Shape& s, const void* ot, const float* rho, const void* gate,
                         bool channel, const void* dy, void* dot, void* dgate, float* part,
                         hipStream_t st);
int launch_head_prenorm_bwd(const Shape& s, const void* q, const void* k, const void* r,
                            const float* tau, void* dq, void* dk, void* dr, float* part,
                            float norm_eps, hipStream_t st);
int launch_head_reduce(const Shape& s, const float* part, float* out, hipStream_t st);

// orthogonal random-feature bank (bank.hip)
int launch_feature_bank(int H, int m, int D, const float* gauss, const float* radii, float* omega,
                        int sign_correct, hipStream_t st);

// (sequence, head) pairs of one decode call: one 256-thread workgroup each on
// a one-dimensional grid (fewer than 2^32 threads)
constexpr int64_t kMaxDecodeGroups = ((int64_t)1 << 24) - 1;

void set_error(const char* fmt, ...);
bool shape_supported(const Shape& s, bool backward);

}  // namespace linsimp
