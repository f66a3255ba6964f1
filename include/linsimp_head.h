/*
 * linsimp_head.h -- C ABI of one full LinSimp attention head: the core of
 * linsimp.h with the steps the paper puts either side of it.
 *
 *   q' = tau_h q / |q|,  k' = k / |k|,  r' = r / |r|       Sec. 3.1 (unit streams, per-head
 *                                                          temperature on the query)
 *   o~ = core(q', k', v, r', u)                             Sec. 3.2-3.3 (linsimp_fwd)
 *   y  = g * RMSNorm(o~),  g = sigmoid(gamma_h)             eq:gated-output (per-head gate)
 *   y  = g_i (*) RMSNorm(o~_i),  g_i = sigmoid(l_i)          Sec. 3.3 (channel-wise,
 *                                                          input-dependent gate)
 *
 * with |x| floored at opts->norm_eps (below it the map is x / norm_eps) and
 * RMSNorm(x) = x / sqrt(mean(x^2) + opts->rms_eps), no learned scale.  For the
 * channel-wise gate the caller passes the projected logits l = W_g x + b_g
 * (the projection belongs to the surrounding model).
 *
 * Conventions are those of linsimp.h: device pointers owned by the caller,
 * 16-byte aligned, dense row-major; the library never allocates; calls only
 * enqueue on `stream`; the return value is LINSIMP_OK or a negative
 * linsimp_status with linsimp_last_error() set.  Shapes: the core's shape
 * support (linsimp.h) with D, Dv in {32, 64, 128}.
 */
#ifndef LINSIMP_HEAD_H
#define LINSIMP_HEAD_H

#include "linsimp.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LINSIMP_GATE_HEAD = 0,     /* gate: float gamma[H];  g = sigmoid(gamma_h)           */
  LINSIMP_GATE_CHANNEL = 1   /* gate: logits [B, H, n, Dv] in dims->dtype; g = sigmoid */
} linsimp_gate_kind;

typedef struct {
  float norm_eps;   /* floor of |x| in the L2 normalisation (1e-12)  */
  float rms_eps;    /* RMSNorm epsilon (1e-6)                         */
  int32_t gate;     /* linsimp_gate_kind                              */
} linsimp_head_opts;

/* Bytes of the `saved` buffer linsimp_head_fwd fills and linsimp_head_bwd
 * reads (normalised q', k', r', the core output o~, its per-row statistics
 * and the RMSNorm factors).  0 for invalid or unsupported dims. */
size_t linsimp_head_saved_size(const linsimp_dims* dims);

/* Bytes of workspace for linsimp_head_fwd (for_backward = 0) or
 * linsimp_head_bwd (for_backward = 1).  0 for invalid or unsupported dims. */
size_t linsimp_head_workspace_size(const linsimp_dims* dims, int for_backward);

/* Forward of the head.
 *   q, k, r : [B, H, n, D] dtype (raw streams)   v, u : [B, H, n, Dv] dtype
 *   omega   : [H, m, D] float32                  tau  : [H] float32
 *   gate    : float gamma[H] (LINSIMP_GATE_HEAD) or logits [B, H, n, Dv] dtype
 *   y       : [B, H, n, Dv] dtype, written
 *   saved   : linsimp_head_saved_size(dims) bytes, 256-byte aligned, written;
 *             pass it unchanged to linsimp_head_bwd.
 * Workspace (linsimp_head_workspace_size(dims, 0)) is scratch. */
int linsimp_head_fwd(const linsimp_dims* dims, const linsimp_head_opts* opts, const void* q,
                     const void* k, const void* v, const void* r, const void* u,
                     const float* omega, const float* tau, const void* gate, void* y, void* saved,
                     size_t saved_bytes, void* workspace, size_t workspace_bytes, void* stream);

/* Backward of the head: exact gradient of sum(dy * y).
 *   q, k, v, r, u, omega, tau, gate : as passed to linsimp_head_fwd
 *   saved : what linsimp_head_fwd wrote for these inputs
 *   dy    : [B, H, n, Dv] dtype
 *   dq, dk, dr : [B, H, n, D] dtype; dv, du : [B, H, n, Dv] dtype; overwritten
 *   dtau  : [H] float32, overwritten
 *   dgate : float dgamma[H] (LINSIMP_GATE_HEAD) or d logits [B, H, n, Dv] dtype,
 *           overwritten
 * The per-head sums dtau and dgamma are reduced in a fixed order
 * (bitwise reproducible).  Workspace: linsimp_head_workspace_size(dims, 1). */
int linsimp_head_bwd(const linsimp_dims* dims, const linsimp_head_opts* opts, const void* q,
                     const void* k, const void* v, const void* r, const void* u,
                     const float* omega, const float* tau, const void* gate, const void* saved,
                     const void* dy, void* dq, void* dk, void* dv, void* dr, void* du, float* dtau,
                     void* dgate, void* workspace, size_t workspace_bytes, void* stream);

/* linsimp_head_bwd with flags: 0, or LINSIMP_BWD_REUSE_STATES (linsimp.h) when
 * `workspace` is the backward-sized head workspace (linsimp_head_workspace_size
 * (dims, 1)) that the matching linsimp_head_fwd call used and nothing has
 * written since: the core's boundary states are reused, results are bitwise
 * those of linsimp_head_bwd. */
int linsimp_head_bwd_ex(const linsimp_dims* dims, const linsimp_head_opts* opts, const void* q,
                        const void* k, const void* v, const void* r, const void* u,
                        const float* omega, const float* tau, const void* gate, const void* saved,
                        const void* dy, void* dq, void* dk, void* dv, void* dr, void* du,
                        float* dtau, void* dgate, int32_t flags, void* workspace,
                        size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LINSIMP_HEAD_H */
