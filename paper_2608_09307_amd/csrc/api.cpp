// C ABI of the LinSimp library: argument validation, workspace carving and
// dispatch to the HIP kernels.  Declarations and contracts: include/linsimp.h
// (the core), include/linsimp_head.h (the full head around it) and
// include/linsimp_bank.h (the feature-bank sampler).
#include "../../include/linsimp.h"
#include "../../include/linsimp_bank.h"
#include "../../include/linsimp_head.h"

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "linsimp_internal.h"
#include "prof.h"

#include <atomic>
#include <mutex>
#include <string>
#include <vector>

namespace linsimp {

static thread_local char g_err[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

static size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

size_t workspace_bytes(const Shape& s, bool backward) {
  const size_t H = (size_t)s.H, BH = (size_t)s.BH(), nch = (size_t)s.nch();
  const size_t md = (size_t)s.m * s.D, S = (size_t)s.state_elems();
  size_t t = 0;
  t += al(H * md * s.esize());                 // omq
  t += al(H * md * 4);                         // omk (bf16 hi+lo, or f32)
  t += al(H * md * 2);                         // omh
  t += al(BH * nch * S * 4);                   // states
  if (s.esize() == 2) t += al(BH * nch * (size_t)s.m * s.Dv * 2);   // states16
  t += al(BH * nch * 4);                       // rho
  t += al(BH * (nch + 1) * 4);                 // rex
  t += al(BH * (size_t)s.n * s.m * s.esize()); // chi
  t += al(BH * (size_t)s.n * 4);               // rj
  if (s.m > 128) t += al((size_t)(s.m / 128) * BH * s.n * (s.Dv + 2) * 4);   // part
  if (backward) {
    const size_t n = (size_t)s.n, nfb = (size_t)bwd_nfb(s.m), ns = (size_t)bwd_slots(s.w);
    t += al(BH * nch * S * 4);                 // gstates
    t += al(BH * n * s.m * 4);                 // dchi
    const size_t nfp = nfb > 1 ? nfb : 0;      // float32 du / dr partials only when m > 128
    t += al(nfb * BH * n * s.Dv * 4);          // dvin
    t += al(nfp * BH * n * s.Dv * 4);          // du32
    t += al(nfp * BH * n * s.D * 4);           // dr32
    t += al(nfb * ns * BH * n * s.D * 4);      // dq32
    t += al(BH * n * 2 * 4);                   // rowstat
  }
  return t;
}

void carve(const Shape& s, void* base, bool backward, Workspace* ws) {
  const size_t H = (size_t)s.H, BH = (size_t)s.BH(), nch = (size_t)s.nch();
  const size_t md = (size_t)s.m * s.D, S = (size_t)s.state_elems();
  char* p = (char*)base;
  memset(ws, 0, sizeof(*ws));
  ws->omq = p; p += al(H * md * s.esize());
  ws->omk = p; p += al(H * md * 4);
  ws->omh = p; p += al(H * md * 2);
  ws->states = (float*)p; p += al(BH * nch * S * 4);
  if (s.esize() == 2) { ws->states16 = p; p += al(BH * nch * (size_t)s.m * s.Dv * 2); }
  ws->rho = (float*)p; p += al(BH * nch * 4);
  ws->rex = (float*)p; p += al(BH * (nch + 1) * 4);
  ws->chi = p; p += al(BH * (size_t)s.n * s.m * s.esize());
  ws->rj = (float*)p; p += al(BH * (size_t)s.n * 4);
  if (s.m > 128) { ws->part = (float*)p; p += al((size_t)(s.m / 128) * BH * s.n * (s.Dv + 2) * 4); }
  if (backward) {
    const size_t n = (size_t)s.n, nfb = (size_t)bwd_nfb(s.m), ns = (size_t)bwd_slots(s.w);
    ws->gstates = (float*)p; p += al(BH * nch * S * 4);
    ws->dchi = (float*)p; p += al(BH * n * s.m * 4);
    const size_t nfp = nfb > 1 ? nfb : 0;
    ws->dvin = (float*)p; p += al(nfb * BH * n * s.Dv * 4);
    ws->du32 = nfp ? (float*)p : nullptr; p += al(nfp * BH * n * s.Dv * 4);
    ws->dr32 = nfp ? (float*)p : nullptr; p += al(nfp * BH * n * s.D * 4);
    ws->dq32 = (float*)p; p += al(nfb * ns * BH * n * s.D * 4);
    ws->rowstat = (float*)p; p += al(BH * n * 2 * 4);
  }
}

// ---- per-kernel timing ----
struct TimedLaunch {
  std::string name;
  hipEvent_t ev0, ev1;
  bool open;        // begin recorded, end not yet
};
static std::mutex g_tmu;
static std::atomic<bool> g_timing{false};
static std::vector<TimedLaunch> g_launches;
static std::vector<hipEvent_t> g_free;

bool timing_on() { return g_timing; }

static hipEvent_t take_event() {
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void timing_mark(const char* name, hipStream_t st, bool begin) {
  std::lock_guard<std::mutex> lk(g_tmu);
  if (begin) {
    TimedLaunch t;
    t.name = name;
    t.ev0 = take_event();
    t.ev1 = take_event();
    if (t.ev0 == nullptr || t.ev1 == nullptr) {     // not timed; keep what was obtained
      if (t.ev0 != nullptr) g_free.push_back(t.ev0);
      if (t.ev1 != nullptr) g_free.push_back(t.ev1);
      return;
    }
    t.open = true;
    hipEventRecord(t.ev0, st);
    g_launches.push_back(t);
  } else {
    // the most recent open launch of this name (scopes of one name never nest)
    for (auto it = g_launches.rbegin(); it != g_launches.rend(); ++it)
      if (it->open && it->name == name) {
        hipEventRecord(it->ev1, st);
        it->open = false;
        break;
      }
  }
}

// ---- which forward's states a workspace holds ----
// linsimp_bwd_ex with LINSIMP_BWD_REUSE_STATES reads the feature-bank copies,
// boundary states, frames and key features a forward left in the workspace.
// Those depend on the dims and on k, v and omega only, so every call that
// writes them records (dims, k, v, omega) under the workspace pointer, calls
// that overwrite them with something else drop the record, and a reusing
// backward is refused unless the record matches its own arguments.
struct StateRecord {
  const void* ws;
  int64_t B, H, n;
  int D, Dv, m, w, dtype;
  const void *k, *v, *omega;
};
static std::mutex g_recmu;
static std::vector<StateRecord> g_records;       // most recent last
static constexpr size_t kMaxRecords = 256;

static void forget_states(const void* ws) {
  std::lock_guard<std::mutex> lk(g_recmu);
  for (size_t i = 0; i < g_records.size(); ++i)
    if (g_records[i].ws == ws) { g_records.erase(g_records.begin() + i); break; }
}

void record_states(const void* ws, const Shape& s, const void* k, const void* v, const void* omega) {
  forget_states(ws);
  std::lock_guard<std::mutex> lk(g_recmu);
  if (g_records.size() >= kMaxRecords) g_records.erase(g_records.begin());
  g_records.push_back(StateRecord{ws, s.B, s.H, s.n, s.D, s.Dv, s.m, s.w, s.dtype, k, v, omega});
}

void drop_states(const void* ws) { forget_states(ws); }

// LINSIMP_OK if `ws` holds the states of a forward with these dims, k, v and omega
int check_states(const void* ws, const Shape& s, const void* k, const void* v, const void* omega) {
  std::lock_guard<std::mutex> lk(g_recmu);
  for (const StateRecord& r : g_records) {
    if (r.ws != ws) continue;
    if (r.B != s.B || r.H != s.H || r.n != s.n || r.D != s.D || r.Dv != s.Dv || r.m != s.m ||
        r.w != s.w || r.dtype != s.dtype) {
      set_error("LINSIMP_BWD_REUSE_STATES: the workspace holds the states of a forward with other dims");
      return LINSIMP_E_INVALID_ARG;
    }
    if (r.k != k || r.v != v || r.omega != omega) {
      set_error("LINSIMP_BWD_REUSE_STATES: the workspace holds the states of a forward with other k, v or omega");
      return LINSIMP_E_INVALID_ARG;
    }
    return LINSIMP_OK;
  }
  set_error("LINSIMP_BWD_REUSE_STATES: no forward has left its states in this workspace "
            "(or a later call overwrote them)");
  return LINSIMP_E_INVALID_ARG;
}

bool shape_supported(const Shape& s, bool /*backward*/) {
  if (s.w < 1 || s.w > 128) return false;
  if (!wide_window_ok(s.dtype, s.D, s.m, (s.w + 31) / 32)) return false;
  if (s.w * (s.m < 128 ? s.m : 128) > 8192 && s.w > 64) return false;
  return fwd_combo_supported(s.dtype, s.D, s.Dv, s.m);
}

}  // namespace linsimp

using namespace linsimp;

static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// Validates dims; fills `s`.  Returns LINSIMP_OK or an error status.
static int check_dims(const linsimp_dims* d, Shape* s, bool backward, bool bh_on_grid_y = true) {
  if (d == nullptr) { set_error("dims is NULL"); return LINSIMP_E_INVALID_ARG; }
  if (d->B < 1 || d->H < 1 || d->n < 1 || d->D < 1 || d->Dv < 1 || d->m < 1 || d->w < 1) {
    set_error("dims must be positive (B=%lld H=%lld n=%lld D=%d Dv=%d m=%d w=%d)",
              (long long)d->B, (long long)d->H, (long long)d->n, d->D, d->Dv, d->m, d->w);
    return LINSIMP_E_INVALID_ARG;
  }
  if (d->dtype != LINSIMP_F32 && d->dtype != LINSIMP_BF16) {
    set_error("dtype %d is not LINSIMP_F32 or LINSIMP_BF16", d->dtype);
    return LINSIMP_E_INVALID_ARG;
  }
  if (!(d->eps >= 0.0f)) { set_error("eps must be >= 0"); return LINSIMP_E_INVALID_ARG; }
  // (batch, head) pairs index the grid's y dimension (not in decode); rows bound the 1-D grids
  if (d->n > (int64_t)1 << 30 || (bh_on_grid_y && d->B * d->H > 65535) ||
      d->B * d->H * d->n > (int64_t)1 << 31) {
    set_error("sizes too large: B*H=%lld (at most 65535), B*H*n=%lld (at most 2^31)",
              (long long)(d->B * d->H), (long long)(d->B * d->H * d->n));
    return LINSIMP_E_UNSUPPORTED;
  }
  s->B = d->B; s->H = d->H; s->n = d->n; s->D = d->D; s->Dv = d->Dv; s->m = d->m; s->w = d->w;
  s->dtype = d->dtype; s->eps = d->eps;
  if (!shape_supported(*s, backward)) {
    set_error("unsupported shape: dtype=%d D=%d Dv=%d m=%d w=%d", d->dtype, d->D, d->Dv, d->m, d->w);
    return LINSIMP_E_UNSUPPORTED;
  }
  return LINSIMP_OK;
}

// the decode kernels run one 256-thread workgroup per (sequence, head) on a
// one-dimensional grid, whose thread count must stay below 2^32
static int check_decode_grid(int64_t S, int32_t H) {
  if (S * (int64_t)H > kMaxDecodeGroups) {
    set_error("decode: S*H = %lld (sequence, head) pairs, at most %lld per call",
              (long long)(S * (int64_t)H), (long long)kMaxDecodeGroups);
    return LINSIMP_E_UNSUPPORTED;
  }
  return LINSIMP_OK;
}

static int check_ptrs(const char* names, const void* const* ps, int np) {
  for (int i = 0; i < np; ++i) {
    if (ps[i] == nullptr) {
      set_error("argument %d of (%s) is NULL", i, names);
      return LINSIMP_E_INVALID_ARG;
    }
    if (!aligned16(ps[i])) {
      set_error("argument %d of (%s) is not 16-byte aligned", i, names);
      return LINSIMP_E_INVALID_ARG;
    }
  }
  return LINSIMP_OK;
}

static int check_ws(const Shape& s, bool backward, const void* ws, size_t bytes) {
  size_t need = workspace_bytes(s, backward);
  if (ws == nullptr || ((uintptr_t)ws & 255) != 0) {
    set_error("workspace must be a non-NULL 256-byte aligned device pointer");
    return LINSIMP_E_WORKSPACE;
  }
  if (bytes < need) {
    set_error("workspace too small: %zu bytes given, %zu needed", bytes, need);
    return LINSIMP_E_WORKSPACE;
  }
  return LINSIMP_OK;
}

extern "C" {

size_t linsimp_workspace_size(const linsimp_dims* dims, int for_backward) {
  Shape s;
  if (check_dims(dims, &s, for_backward != 0) != LINSIMP_OK) return 0;
  return workspace_bytes(s, for_backward != 0);
}

int linsimp_fwd(const linsimp_dims* dims, const void* q, const void* k, const void* v,
                const void* r, const void* u, const float* omega, void* out, float* stats,
                void* workspace, size_t workspace_bytes_, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s, false);
  if (rc) return rc;
  const void* ps[] = {q, k, v, r, u, omega, out};
  if ((rc = check_ptrs("q,k,v,r,u,omega,out", ps, 7))) return rc;
  if (stats != nullptr && !aligned16(stats)) {
    set_error("stats is not 16-byte aligned");
    return LINSIMP_E_INVALID_ARG;
  }
  if ((rc = check_ws(s, false, workspace, workspace_bytes_))) return rc;
  Workspace ws;
  carve(s, workspace, false, &ws);
  rc = launch_forward(s, q, k, v, r, u, omega, out, stats, nullptr, nullptr, nullptr, ws,
                      (hipStream_t)stream);
  if (rc == LINSIMP_OK) record_states(workspace, s, k, v, omega);
  else drop_states(workspace);
  return rc;
}

int linsimp_bwd(const linsimp_dims* dims, const void* q, const void* k, const void* v,
                const void* r, const void* u, const float* omega, const void* out,
                const float* stats, const void* dout, void* dq, void* dk, void* dv, void* dr,
                void* du, void* workspace, size_t workspace_bytes_, void* stream) {
  return linsimp_bwd_ex(dims, q, k, v, r, u, omega, out, stats, dout, dq, dk, dv, dr, du, 0, workspace,
                        workspace_bytes_, stream);
}

int linsimp_bwd_ex(const linsimp_dims* dims, const void* q, const void* k, const void* v,
                   const void* r, const void* u, const float* omega, const void* out,
                   const float* stats, const void* dout, void* dq, void* dk, void* dv, void* dr,
                   void* du, int32_t flags, void* workspace, size_t workspace_bytes_, void* stream) {
  if (flags != 0 && flags != LINSIMP_BWD_REUSE_STATES) {
    set_error("bwd flags %d: only 0 or LINSIMP_BWD_REUSE_STATES", flags);
    return LINSIMP_E_INVALID_ARG;
  }
  Shape s;
  int rc = check_dims(dims, &s, true);
  if (rc) return rc;
  const void* ps[] = {q, k, v, r, u, omega, out, stats, dout, dq, dk, dv, dr, du};
  if ((rc = check_ptrs("q,k,v,r,u,omega,out,stats,dout,dq,dk,dv,dr,du", ps, 14))) return rc;
  if ((rc = check_ws(s, true, workspace, workspace_bytes_))) return rc;
  const bool reuse = flags == LINSIMP_BWD_REUSE_STATES;
  if (reuse && (rc = check_states(workspace, s, k, v, omega))) return rc;
  Workspace ws;
  carve(s, workspace, true, &ws);
  rc = launch_backward(s, q, k, v, r, u, omega, out, stats, dout, dq, dk, dv, dr, du, ws,
                       (hipStream_t)stream, reuse);
  // without reuse the backward re-ran the forward's state passes on its inputs
  if (rc == LINSIMP_OK) { if (!reuse) record_states(workspace, s, k, v, omega); }
  else drop_states(workspace);
  return rc;
}

int linsimp_prefill(const linsimp_dims* dims, const void* k, const void* v, const void* r,
                    const void* u, const float* omega, float* M, float* a, float* rho,
                    void* ring_r, void* ring_u, int64_t* pos, void* workspace,
                    size_t workspace_bytes_, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s, false);
  if (rc) return rc;
  const void* ps[] = {k, v, r, u, omega, M, a, rho, ring_r, ring_u, pos};
  if ((rc = check_ptrs("k,v,r,u,omega,M,a,rho,ring_r,ring_u,pos", ps, 11))) return rc;
  if ((rc = check_ws(s, false, workspace, workspace_bytes_))) return rc;
  Workspace ws;
  carve(s, workspace, false, &ws);
  drop_states(workspace);          // the prefill leaves no reusable forward states
  rc = launch_forward(s, k, k, v, r, u, omega, nullptr, nullptr, M, a, rho, ws, (hipStream_t)stream);
  if (rc) return rc;
  return launch_ring_fill(s, r, u, ring_r, ring_u, pos, (hipStream_t)stream);
}

int linsimp_decode_step(int64_t S, int32_t H, int32_t D, int32_t Dv, int32_t m, int32_t w,
                        int32_t dtype, float eps, const void* q, const void* k, const void* v,
                        const void* r, const void* u, const float* omega, float* M, float* a,
                        float* rho, void* ring_r, void* ring_u, int64_t* pos, void* out,
                        void* stream) {
  linsimp_dims d;
  d.B = S; d.H = H; d.n = 1; d.D = D; d.Dv = Dv; d.m = m; d.w = w; d.dtype = dtype; d.eps = eps;
  Shape s;
  int rc = check_dims(&d, &s, false, false);
  if (rc) return rc;
  if ((rc = check_decode_grid(S, H))) return rc;
  const void* ps[] = {q, k, v, r, u, omega, M, a, rho, ring_r, ring_u, pos, out};
  if ((rc = check_ptrs("q,k,v,r,u,omega,M,a,rho,ring_r,ring_u,pos,out", ps, 13))) return rc;
  return launch_decode(S, H, 1, D, Dv, m, w, dtype, eps, q, k, v, r, u, omega, M, a, rho, ring_r,
                       ring_u, pos, out, (hipStream_t)stream);
}

int linsimp_decode_chunk(int64_t S, int32_t H, int32_t T, int32_t D, int32_t Dv, int32_t m,
                         int32_t w, int32_t dtype, float eps, const void* q, const void* k,
                         const void* v, const void* r, const void* u, const float* omega, float* M,
                         float* a, float* rho, void* ring_r, void* ring_u, int64_t* pos, void* out,
                         void* stream) {
  if (T < 1 || T > 4096) {
    set_error("decode_chunk: T=%d not in [1, 4096]", T);
    return LINSIMP_E_INVALID_ARG;
  }
  linsimp_dims d;
  d.B = S; d.H = H; d.n = T; d.D = D; d.Dv = Dv; d.m = m; d.w = w; d.dtype = dtype; d.eps = eps;
  Shape s;
  int rc = check_dims(&d, &s, false, false);
  if (rc) return rc;
  if ((rc = check_decode_grid(S, H))) return rc;
  const void* ps[] = {q, k, v, r, u, omega, M, a, rho, ring_r, ring_u, pos, out};
  if ((rc = check_ptrs("q,k,v,r,u,omega,M,a,rho,ring_r,ring_u,pos,out", ps, 13))) return rc;
  return launch_decode(S, H, T, D, Dv, m, w, dtype, eps, q, k, v, r, u, omega, M, a, rho, ring_r,
                       ring_u, pos, out, (hipStream_t)stream);
}

int linsimp_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = on != 0;
  return LINSIMP_OK;
}

int linsimp_timing_read(char* names, int names_len, float* total_ms, int* counts, int max_kernels) {
  std::lock_guard<std::mutex> lk(g_tmu);
  if (names == nullptr || total_ms == nullptr || counts == nullptr || names_len < 1 || max_kernels < 1) {
    set_error("timing_read: bad output buffers");
    return LINSIMP_E_INVALID_ARG;
  }
  std::vector<std::string> keys;
  std::vector<double> tot;
  std::vector<int> cnt;
  int rc = LINSIMP_OK;
  for (auto& t : g_launches) {
    if (t.open) continue;                             // its end was never marked
    if (hipEventSynchronize(t.ev1) != hipSuccess) { rc = LINSIMP_E_HIP; continue; }
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, t.ev0, t.ev1) != hipSuccess) { rc = LINSIMP_E_HIP; continue; }
    size_t k = 0;
    while (k < keys.size() && keys[k] != t.name) ++k;
    if (k == keys.size()) { keys.push_back(t.name); tot.push_back(0.0); cnt.push_back(0); }
    tot[k] += ms;
    cnt[k] += 1;
  }
  for (auto& t : g_launches) { g_free.push_back(t.ev0); g_free.push_back(t.ev1); }
  g_launches.clear();
  std::string all;
  int nk = 0;
  // only whole names that fit the caller's buffer (with its terminating NUL)
  for (size_t k = 0; k < keys.size() && nk < max_kernels; ++k, ++nk) {
    if (all.size() + keys[k].size() + 1 >= (size_t)names_len) break;
    all += keys[k];
    all += '\n';
    total_ms[nk] = (float)tot[k];
    counts[nk] = cnt[k];
  }
  snprintf(names, (size_t)names_len, "%s", all.c_str());
  if (rc != LINSIMP_OK) set_error("timing_read: a HIP event query failed");
  return rc < 0 ? rc : nk;
}

}  // extern "C"

// ---- forward without a caller workspace (linsimp_fwd_static) ----
// Its scratch is this file-scope device array: each GPU the library runs on
// holds one copy, allocated with the code object, until the process ends.  In
// host code `scratch` names a host-side stand-in, not a device address; the
// address of the current device's copy comes from hipGetSymbolAddress, once
// per device with that device current, and only that pointer is handed to
// kernels.
static __device__ __align__(256) unsigned char scratch[LINSIMP_FWD_STATIC_MAX_BYTES];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scr_mu;
void* g_scr_ptr[kMaxScratchDevices] = {};

int current_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) {
    set_error("fwd_static: no usable current device (%s)", hipGetErrorString(e));
    return LINSIMP_E_HIP;
  }
  std::lock_guard<std::mutex> lk(g_scr_mu);
  if (g_scr_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      set_error("fwd_static: address of the static scratch on device %d: %s", dev, hipGetErrorString(e));
      return LINSIMP_E_HIP;
    }
    g_scr_ptr[dev] = p;
  }
  *out = g_scr_ptr[dev];
  return LINSIMP_OK;
}

}  // namespace

extern "C" {

int linsimp_fwd_static(const linsimp_dims* dims, const void* q, const void* k, const void* v,
                       const void* r, const void* u, const float* omega, void* out, float* stats,
                       void* stream) {
  Shape s;
  int rc = check_dims(dims, &s, false);
  if (rc) return rc;
  const void* ps[] = {q, k, v, r, u, omega, out};
  if ((rc = check_ptrs("q,k,v,r,u,omega,out", ps, 7))) return rc;
  if (stats != nullptr && !aligned16(stats)) {
    set_error("stats is not 16-byte aligned");
    return LINSIMP_E_INVALID_ARG;
  }
  const size_t need = workspace_bytes(s, false);
  if (need > (size_t)LINSIMP_FWD_STATIC_MAX_BYTES) {
    set_error("fwd_static: these dims need %zu bytes of scratch; the static scratch holds %zu "
              "(use linsimp_fwd with a workspace)", need, (size_t)LINSIMP_FWD_STATIC_MAX_BYTES);
    return LINSIMP_E_WORKSPACE;
  }
  void* base = nullptr;
  if ((rc = current_scratch(&base))) return rc;
  Workspace ws;
  carve(s, base, false, &ws);
  return launch_forward(s, q, k, v, r, u, omega, out, stats, nullptr, nullptr, nullptr, ws,
                        (hipStream_t)stream);
}

// ---- full head (include/linsimp_head.h) ----
}  // extern "C"

namespace {

// `saved` of the head: q', k', r' [BH n D], o~ [BH n Dv] (dtype), stats [BH n 2]
// and rho [BH n] (float32), each region 256-byte aligned.
struct HeadSaved {
  void *qn, *kn, *rn, *ot;
  float *stats, *rho;
};

size_t head_saved_bytes(const Shape& s, HeadSaved* hs, void* base) {
  const size_t rows = (size_t)s.BH() * s.n;
  const size_t es = s.esize();
  size_t off = 0;
  auto take = [&](size_t bytes) {
    void* p = base ? (char*)base + off : nullptr;
    off += al(bytes);
    return p;
  };
  void* qn = take(rows * s.D * es);
  void* kn = take(rows * s.D * es);
  void* rn = take(rows * s.D * es);
  void* ot = take(rows * s.Dv * es);
  float* stats = (float*)take(rows * 2 * sizeof(float));
  float* rho = (float*)take(rows * sizeof(float));
  if (hs) *hs = HeadSaved{qn, kn, rn, ot, stats, rho};
  return off;
}

// backward workspace: the core's, then d o~ [BH n Dv] dtype and the per-row
// partials [BH n] float32 of dgamma and dtau
size_t head_ws_bytes(const Shape& s, bool backward) {
  size_t b = al(workspace_bytes(s, backward));
  if (backward) {
    const size_t rows = (size_t)s.BH() * s.n;
    b += al(rows * s.Dv * s.esize()) + 2 * al(rows * sizeof(float));
  }
  return b;
}

int check_head(const linsimp_dims* dims, const linsimp_head_opts* opts, Shape* s, bool backward) {
  int rc = check_dims(dims, s, backward);
  if (rc) return rc;
  if (opts == nullptr) { set_error("opts is NULL"); return LINSIMP_E_INVALID_ARG; }
  if (opts->gate != LINSIMP_GATE_HEAD && opts->gate != LINSIMP_GATE_CHANNEL) {
    set_error("opts->gate %d is not a linsimp_gate_kind", opts->gate);
    return LINSIMP_E_INVALID_ARG;
  }
  if (!(opts->norm_eps > 0.0f) || !(opts->rms_eps >= 0.0f)) {
    set_error("opts: norm_eps must be > 0 and rms_eps >= 0");
    return LINSIMP_E_INVALID_ARG;
  }
  const bool okw = (s->D == 32 || s->D == 64 || s->D == 128) && (s->Dv == 32 || s->Dv == 64 || s->Dv == 128);
  if (!okw) {
    set_error("head: D=%d Dv=%d not in {32, 64, 128}", s->D, s->Dv);
    return LINSIMP_E_UNSUPPORTED;
  }
  return LINSIMP_OK;
}

int check_buf(const char* what, const void* p, size_t bytes, size_t need) {
  if (p == nullptr || ((uintptr_t)p & 255) != 0) {
    set_error("%s must be a non-NULL 256-byte aligned device pointer", what);
    return LINSIMP_E_WORKSPACE;
  }
  if (bytes < need) {
    set_error("%s too small: %zu bytes given, %zu needed", what, bytes, need);
    return LINSIMP_E_WORKSPACE;
  }
  return LINSIMP_OK;
}

}  // namespace

extern "C" {

size_t linsimp_head_saved_size(const linsimp_dims* dims) {
  Shape s;
  linsimp_head_opts o{1e-12f, 1e-6f, LINSIMP_GATE_HEAD};
  if (check_head(dims, &o, &s, false) != LINSIMP_OK) return 0;
  return head_saved_bytes(s, nullptr, nullptr);
}

size_t linsimp_head_workspace_size(const linsimp_dims* dims, int for_backward) {
  Shape s;
  linsimp_head_opts o{1e-12f, 1e-6f, LINSIMP_GATE_HEAD};
  if (check_head(dims, &o, &s, for_backward != 0) != LINSIMP_OK) return 0;
  return head_ws_bytes(s, for_backward != 0);
}

int linsimp_head_fwd(const linsimp_dims* dims, const linsimp_head_opts* opts, const void* q,
                     const void* k, const void* v, const void* r, const void* u,
                     const float* omega, const float* tau, const void* gate, void* y, void* saved,
                     size_t saved_bytes, void* workspace, size_t workspace_bytes_, void* stream) {
  Shape s;
  int rc = check_head(dims, opts, &s, false);
  if (rc) return rc;
  const void* ps[] = {q, k, v, r, u, omega, tau, gate, y};
  if ((rc = check_ptrs("q,k,v,r,u,omega,tau,gate,y", ps, 9))) return rc;
  if ((rc = check_buf("saved", saved, saved_bytes, head_saved_bytes(s, nullptr, nullptr)))) return rc;
  if ((rc = check_buf("workspace", workspace, workspace_bytes_, head_ws_bytes(s, false)))) return rc;
  hipStream_t st = (hipStream_t)stream;
  HeadSaved hs;
  head_saved_bytes(s, &hs, saved);
  Workspace ws;
  carve(s, workspace, false, &ws);
  drop_states(workspace);
  if ((rc = launch_head_prenorm(s, q, k, r, tau, hs.qn, hs.kn, hs.rn, opts->norm_eps, st))) return rc;
  if ((rc = launch_forward(s, hs.qn, hs.kn, v, hs.rn, u, omega, hs.ot, hs.stats, nullptr, nullptr,
                           nullptr, ws, st)))
    return rc;
  // the core's states are those of the normalised keys in `saved`
  record_states(workspace, s, hs.kn, v, omega);
  return launch_head_gate(s, hs.ot, gate, opts->gate == LINSIMP_GATE_CHANNEL, y, hs.rho,
                          opts->rms_eps, st);
}

int linsimp_head_bwd(const linsimp_dims* dims, const linsimp_head_opts* opts, const void* q,
                     const void* k, const void* v, const void* r, const void* u,
                     const float* omega, const float* tau, const void* gate, const void* saved,
                     const void* dy, void* dq, void* dk, void* dv, void* dr, void* du, float* dtau,
                     void* dgate, void* workspace, size_t workspace_bytes_, void* stream) {
  return linsimp_head_bwd_ex(dims, opts, q, k, v, r, u, omega, tau, gate, saved, dy, dq, dk, dv, dr, du,
                             dtau, dgate, 0, workspace, workspace_bytes_, stream);
}

int linsimp_head_bwd_ex(const linsimp_dims* dims, const linsimp_head_opts* opts, const void* q,
                        const void* k, const void* v, const void* r, const void* u,
                        const float* omega, const float* tau, const void* gate, const void* saved,
                        const void* dy, void* dq, void* dk, void* dv, void* dr, void* du,
                        float* dtau, void* dgate, int32_t flags, void* workspace,
                        size_t workspace_bytes_, void* stream) {
  if (flags != 0 && flags != LINSIMP_BWD_REUSE_STATES) {
    set_error("head bwd flags %d: only 0 or LINSIMP_BWD_REUSE_STATES", flags);
    return LINSIMP_E_INVALID_ARG;
  }
  Shape s;
  int rc = check_head(dims, opts, &s, true);
  if (rc) return rc;
  const void* ps[] = {q, k, v, r, u, omega, tau, gate, dy, dq, dk, dv, dr, du, dtau, dgate};
  if ((rc = check_ptrs("q,k,v,r,u,omega,tau,gate,dy,dq,dk,dv,dr,du,dtau,dgate", ps, 16))) return rc;
  if (saved == nullptr || ((uintptr_t)saved & 255) != 0) {
    set_error("saved must be the 256-byte aligned buffer linsimp_head_fwd filled");
    return LINSIMP_E_INVALID_ARG;
  }
  if ((rc = check_buf("workspace", workspace, workspace_bytes_, head_ws_bytes(s, true)))) return rc;
  hipStream_t st = (hipStream_t)stream;
  const bool channel = opts->gate == LINSIMP_GATE_CHANNEL;
  const bool reuse = flags == LINSIMP_BWD_REUSE_STATES;
  HeadSaved hs;
  head_saved_bytes(s, &hs, (void*)saved);
  if (reuse && (rc = check_states(workspace, s, hs.kn, v, omega))) return rc;
  Workspace ws;
  carve(s, workspace, true, &ws);
  const size_t rows = (size_t)s.BH() * s.n;
  char* tail = (char*)workspace + al(workspace_bytes(s, true));
  void* dot = tail;
  float* part_g = (float*)(tail + al(rows * s.Dv * s.esize()));
  float* part_t = (float*)((char*)part_g + al(rows * sizeof(float)));
  if ((rc = launch_head_gate_bwd(s, hs.ot, hs.rho, gate, channel, dy, dot, dgate, part_g, st))) return rc;
  // core gradients with respect to q', k', r' land in dq, dk, dr and are
  // turned into gradients with respect to q, k, r in place
  if ((rc = launch_backward(s, hs.qn, hs.kn, v, hs.rn, u, omega, hs.ot, hs.stats, dot, dq, dk, dv, dr,
                            du, ws, st, reuse))) {
    drop_states(workspace);
    return rc;
  }
  if (!reuse) record_states(workspace, s, hs.kn, v, omega);
  if ((rc = launch_head_prenorm_bwd(s, q, k, r, tau, dq, dk, dr, part_t, opts->norm_eps, st))) return rc;
  if ((rc = launch_head_reduce(s, part_t, dtau, st))) return rc;
  if (!channel && (rc = launch_head_reduce(s, part_g, (float*)dgate, st))) return rc;
  return LINSIMP_OK;
}

int linsimp_feature_bank(int32_t H, int32_t m, int32_t D, const float* gauss, const float* radii,
                         float* omega, int32_t sign_correct, void* stream) {
  if (H < 1 || m < 1 || D < 1) {
    set_error("feature bank: H, m and D must be positive (H=%d m=%d D=%d)", H, m, D);
    return LINSIMP_E_INVALID_ARG;
  }
  if (D != 32 && D != 64 && D != 128) {
    set_error("feature bank: D=%d not in {32, 64, 128}", D);
    return LINSIMP_E_UNSUPPORTED;
  }
  if (sign_correct != 0 && sign_correct != 1) {
    set_error("feature bank: sign_correct must be 0 or 1");
    return LINSIMP_E_INVALID_ARG;
  }
  if ((int64_t)H * ((m + D - 1) / D) > 65535) {
    set_error("feature bank: H * ceil(m / D) = %lld blocks is above 65535",
              (long long)H * ((m + D - 1) / D));
    return LINSIMP_E_UNSUPPORTED;
  }
  const void* ps[] = {gauss, radii, omega};
  int rc = check_ptrs("gauss,radii,omega", ps, 3);
  if (rc) return rc;
  return launch_feature_bank(H, m, D, gauss, radii, omega, sign_correct, (hipStream_t)stream);
}

const char* linsimp_last_error(void) { return g_err; }

int linsimp_version(void) { return 103; }

}  // extern "C"
