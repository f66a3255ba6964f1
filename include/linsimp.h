/*
 * linsimp.h -- C ABI of the LinSimp (Linearized 2-Simplicial Attention) core
 * for AMD Instinct MI355X (gfx950).
 *
 * The operation (paper: "Linearized 2-Simplicial Attention", Sec. 3.2-3.3;
 * App. A; App. C), for every batch b, head h and 0-based row i = 0..n-1:
 *
 *   phi(x) = m^{-1/2} exp(Omega_h x - |x|^2/2 * 1)          Sec. 3.2, eq:prf
 *   z_ic   = q_i (*) r_c                                     Sec. 3.2 (composite query)
 *   M_i    = sum_{j<=i} phi(k_j) v_j^T,  a_i = sum_{j<=i} phi(k_j)   eq:Mstate, eq:astate
 *   C_i    = {max(0, i-w+1), ..., i}                          Sec. 3.3
 *   N_i    = sum_{c in C_i} [phi(z_ic)^T M_i] (*) u_c          eq:Ni
 *   Z_i    = sum_{c in C_i} phi(z_ic)^T a_i                    eq:Zi
 *   out_i  = N_i / (Z_i + eps)                                 eq:linearized-output
 *
 * q, k, r are used exactly as passed: the caller applies the L2 normalisation
 * and the temperature of Sec. 3.1 (q = tau*q_hat, k = k_hat, r = r_hat) and
 * the gated RMSNorm of eq:gated-output outside this library.  Omega is one
 * [m, D] feature bank per head (App. B.1), float32, not differentiated.
 *
 * Numerics: all exponentials are evaluated in log space with a per-row query
 * shift (App. B.2) and a causal running maximum of the key log features; the
 * shifts cancel in the ratio, and eps is added to Z after both shifts (so eps
 * only matters where the shifted Z underflows).  bf16 inputs are used as
 * matrix-core operands with float32 accumulation and float32 prefix states.
 * For bf16 inputs the composite-query logits run on the f16 matrix cores:
 * q, r (and u in the backward) are converted to f16 and z = q (*) r is
 * formed in f16, so the entries of q, r, u and of q (*) r must stay below
 * f16's largest value (65504) in magnitude; entries below 2^-14 keep fewer
 * bits.  Normalised streams (Sec. 3.1) are far inside that range.  Outside
 * it the rows whose queries or anchors overflow come out non-finite (inf or
 * NaN); no status reports it, since the library never reads tensor data on
 * the host.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers owned by the caller, 16-byte aligned,
 *     dense, row-major, in the layouts stated per argument.  The library never
 *     allocates device memory; scratch comes from the caller's workspace
 *     (256-byte aligned, size from linsimp_workspace_size).
 *   - `stream` is a hipStream_t (may be NULL for the default stream).  Calls
 *     only enqueue work on it; nothing synchronises the device.
 *   - Return value: LINSIMP_OK or a negative linsimp_status; the library never
 *     aborts or throws across the ABI.  linsimp_last_error() gives a message
 *     for the last failure on the calling thread.
 *   - Supported shapes: dtype bf16 with (D = Dv, m) in {(32,32), (64,64),
 *     (64,128), (128,64), (128,128), (128,256)}; dtype f32 with D = Dv in
 *     {32, 64} and m in {32, 64}; 1 <= w <= 64 for every combination, and
 *     64 < w <= 128 where w * m <= 8192 (the launch rule of App. C
 *     "Dispatch": m <= 64 here), except f32 with D = m = 64, which stops at
 *     w = 96; any n >= 1 (tails are masked); B*H <= 65535 (the decode calls
 *     excepted) and B*H*n <= 2^31.
 *     Other shapes return LINSIMP_E_UNSUPPORTED: there is no fallback path.
 */
#ifndef LINSIMP_H
#define LINSIMP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LINSIMP_OK = 0,
  LINSIMP_E_INVALID_ARG = -1,   /* null / misaligned pointer, bad size          */
  LINSIMP_E_UNSUPPORTED = -2,   /* valid but unsupported shape or dtype         */
  LINSIMP_E_WORKSPACE = -3,     /* workspace missing, misaligned or too small   */
  LINSIMP_E_HIP = -4            /* a HIP runtime call or kernel launch failed   */
} linsimp_status;

typedef enum { LINSIMP_F32 = 0, LINSIMP_BF16 = 1 } linsimp_dtype;

typedef struct {
  int64_t B;       /* batch                                   */
  int64_t H;       /* heads                                   */
  int64_t n;       /* sequence length (rows)                  */
  int32_t D;       /* width of q, k, r                        */
  int32_t Dv;      /* width of v, u, out                      */
  int32_t m;       /* feature rank (rows of Omega)            */
  int32_t w;       /* anchor window width                     */
  int32_t dtype;   /* linsimp_dtype of q, k, v, r, u, out, grads */
  float eps;       /* denominator guard, 1e-30 in the paper   */
} linsimp_dims;

/* Bytes of workspace linsimp_fwd (for_backward = 0), linsimp_bwd
 * (for_backward = 1) or linsimp_prefill (for_backward = 0) needs for `dims`.
 * Returns 0 for invalid or unsupported dims. */
size_t linsimp_workspace_size(const linsimp_dims* dims, int for_backward);

/* Forward pass (Sec. 3.3 eq:Ni, eq:Zi, eq:linearized-output; App. C Alg. 1).
 *   q, k, r : [B, H, n, D]  dtype        v, u : [B, H, n, Dv] dtype
 *   omega   : [H, m, D] float32 (the feature bank Omega of each head)
 *   out     : [B, H, n, Dv] dtype, written (the pre-RMSNorm output o~)
 *   stats   : [B, H, n, 2] float32 or NULL; per row (L_i, Zhat_i): the query
 *             log2 shift and the doubly shifted denominator.  linsimp_bwd
 *             needs it (the paper saves one stabiliser per row, Sec. 4.2).
 * Workspace is scratch; its contents after the call are unspecified. */
int linsimp_fwd(const linsimp_dims* dims, const void* q, const void* k, const void* v,
                const void* r, const void* u, const float* omega, void* out, float* stats,
                void* workspace, size_t workspace_bytes, void* stream);

/* linsimp_fwd for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same forward, with its scratch taken from a static array inside the library
 * instead of a caller workspace.  It calls no hipMalloc, hipFree or other
 * allocating routine; each GPU holds one such array of
 * LINSIMP_FWD_STATIC_MAX_BYTES from the library's load on that GPU until the
 * process ends.  Dims whose forward workspace (linsimp_workspace_size(dims, 0))
 * exceeds it return LINSIMP_E_WORKSPACE without launching anything.  The
 * array belongs to the current device, so `stream` must be a stream of that
 * device.  Every call on a GPU uses the same array: calls that overlap on one
 * GPU (on different streams or host threads) race and give undefined results;
 * calls ordered on one stream are safe.  Nothing in the array needs clearing
 * between calls (every byte the forward reads it first writes).  Arguments,
 * results and bits are those of linsimp_fwd. */
#define LINSIMP_FWD_STATIC_MAX_BYTES (64u << 20)
int linsimp_fwd_static(const linsimp_dims* dims, const void* q, const void* k, const void* v,
                       const void* r, const void* u, const float* omega, void* out, float* stats,
                       void* stream);

/* Backward pass: exact gradient of sum_i dout_i . out_i with respect to q, k,
 * v, r, u, with the stabilising shifts treated as constants (they cancel in
 * the ratio, App. B.2); App. C "Backward query sweep" / "Backward state sweep".
 *   q, k, v, r, u, omega : as in linsimp_fwd (same values)
 *   out, stats           : what linsimp_fwd returned for these inputs
 *   dout                 : [B, H, n, Dv] dtype, upstream gradient
 *   dq, dk, dr : [B, H, n, D] dtype; dv, du : [B, H, n, Dv] dtype; overwritten.
 * No gradient is produced for omega (a fixed buffer, App. B.1). */
int linsimp_bwd(const linsimp_dims* dims, const void* q, const void* k, const void* v,
                const void* r, const void* u, const float* omega, const void* out,
                const float* stats, const void* dout, void* dq, void* dk, void* dv, void* dr,
                void* du, void* workspace, size_t workspace_bytes, void* stream);

/* Flags of linsimp_bwd_ex. */
enum {
  /* The workspace is the one the matching linsimp_fwd call used (sized for
   * the backward, linsimp_workspace_size(dims, 1)), with the same dims and
   * inputs, and nothing has written it since: its feature-bank copies,
   * boundary states and key features are reused instead of recomputed (the
   * backward otherwise re-runs the forward's state and key-feature passes).
   * Results are bitwise those of linsimp_bwd.  Those states depend on the
   * dims, k, v and omega only: the library keeps a host-side record of the
   * last call that left states in each workspace (linsimp_fwd, or
   * linsimp_bwd_ex without the flag) and returns LINSIMP_E_INVALID_ARG when
   * the record is missing (no such call, or a later linsimp_prefill or failed
   * call on the same workspace) or names other dims or other k, v or omega
   * pointers.  The contents behind those pointers must not have changed since
   * (the library does not read data on the host). */
  LINSIMP_BWD_REUSE_STATES = 1
};

/* linsimp_bwd with flags (0 or LINSIMP_BWD_REUSE_STATES); otherwise the same
 * contract. */
int linsimp_bwd_ex(const linsimp_dims* dims, const void* q, const void* k, const void* v,
                   const void* r, const void* u, const float* omega, const void* out,
                   const float* stats, const void* dout, void* dq, void* dk, void* dv, void* dr,
                   void* du, int32_t flags, void* workspace, size_t workspace_bytes, void* stream);

/* Prefill: build the decode state of Theorem 1 from a prefix of n tokens
 * (dims->n) per sequence; dims->B is the number of sequences S.
 *   k, r : [S, H, n, D] dtype;  v, u : [S, H, n, Dv] dtype; omega [H, m, D] f32
 *   M    : [S, H, m, Dv] float32 out;  a : [S, H, m] float32 out
 *   rho  : [S, H] float32 out.  The prefix state of eq:Mstate / eq:astate is
 *          M_true = 2^rho * M and a_true = 2^rho * a (rho is a log2 frame that
 *          keeps M finite whatever the key scale).
 *   ring_r : [S, H, w, D], ring_u : [S, H, w, Dv] dtype out: token j of the
 *          last min(n, w) tokens sits in slot j mod w; other slots are zeroed.
 *   pos  : [S] int64 out, set to n. */
int linsimp_prefill(const linsimp_dims* dims, const void* k, const void* v, const void* r,
                    const void* u, const float* omega, float* M, float* a, float* rho,
                    void* ring_r, void* ring_u, int64_t* pos, void* workspace,
                    size_t workspace_bytes, void* stream);

/* One autoregressive decode step (Theorem 1) for S independent sequences:
 * token t = pos[s] of sequence s updates M and a (eq:Mstate, eq:astate),
 * writes (r_t, u_t) into ring slot t mod w, and reads q_t out over the
 * min(t+1, w) most recent anchors, the new token included.  Ring slots that
 * hold no token yet (slots t+1 .. w-1 while t + 1 < w) do not affect the
 * result, whatever they contain.
 *   q, k, r : [S, H, D] dtype;  v, u : [S, H, Dv] dtype;  omega [H, m, D] f32
 *   M, a, rho, ring_r, ring_u, pos : in/out, layouts as in linsimp_prefill
 *   out : [S, H, Dv] dtype
 * Uses no workspace.  Same shape support as the forward; 1 <= S and
 * S*H <= 2^24 - 1 (one workgroup per (sequence, head); more returns
 * LINSIMP_E_UNSUPPORTED).  pos advances only when the step was enqueued. */
int linsimp_decode_step(int64_t S, int32_t H, int32_t D, int32_t Dv, int32_t m, int32_t w,
                        int32_t dtype, float eps, const void* q, const void* k, const void* v,
                        const void* r, const void* u, const float* omega, float* M, float* a,
                        float* rho, void* ring_r, void* ring_u, int64_t* pos, void* out,
                        void* stream);

/* T consecutive decode steps in one call (Theorem 1 applied T times): token j
 * of sequence s is position pos[s] + j; the result equals T calls of
 * linsimp_decode_step.  The state stays on chip for the whole chunk (M, for
 * m <= 128, in registers; the ring and a in LDS/registers), so it is read and
 * written once per call instead of once per token.
 *   q, k, r : [S, H, T, D] dtype;  v, u : [S, H, T, Dv] dtype; omega [H, m, D] f32
 *   M, a, rho, ring_r, ring_u, pos : in/out, layouts as in linsimp_prefill
 *   out : [S, H, T, Dv] dtype
 * 1 <= T <= 4096.  Uses no workspace.  Same shape support and S*H bound as
 * linsimp_decode_step. */
int linsimp_decode_chunk(int64_t S, int32_t H, int32_t T, int32_t D, int32_t Dv, int32_t m,
                         int32_t w, int32_t dtype, float eps, const void* q, const void* k,
                         const void* v, const void* r, const void* u, const float* omega, float* M,
                         float* a, float* rho, void* ring_r, void* ring_u, int64_t* pos, void* out,
                         void* stream);

/* Per-kernel timing, for tuning and roofline reports.  While enabled
 * (on != 0), every kernel the library launches is bracketed by two HIP events
 * recorded on its stream; enabling costs two event records per launch and
 * changes nothing else.  Process-wide; returns LINSIMP_OK. */
int linsimp_timing_enable(int on);

/* Waits for the events recorded since the previous read, sums them per kernel
 * name and clears them.  Writes up to max_kernels entries: names (a
 * newline-separated list, NUL-terminated, into names[names_len]), total_ms[i]
 * (summed milliseconds) and counts[i] (launches).  Returns the number of
 * kernels written (>= 0) or a negative linsimp_status. */
int linsimp_timing_read(char* names, int names_len, float* total_ms, int* counts,
                        int max_kernels);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* linsimp_last_error(void);

/* ABI version (major * 100 + minor). */
int linsimp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LINSIMP_H */
