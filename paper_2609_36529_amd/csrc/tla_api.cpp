// C ABI of the triadic linear attention library: host-side validation,
// workspace carving and the fixed launch sequence of each entry point.
// Validation never touches the device, so a rejected call launches nothing.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <vector>

#include <hip/hip_runtime.h>

#include "../../include/tla.h"
#include "tla_internal.hpp"

// Device scratch of tla_fwd_noalloc: the inference forward's per-chunk
// workspace (coefficient vectors, gamma^C, operand tiles) for callers that
// cannot allocate.  One copy per GPU, held until the process ends.  Host code
// never uses this name as an address: the device address of each GPU's copy
// comes from hipGetSymbolAddress (scratch_ptr below).
static __device__ __align__(256) unsigned char scratch[TLA_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool misaligned(const void* p) { return p && ((uintptr_t)p & 15u) != 0; }

bool pow2_in(int x, const int* set, int n) {
  for (int i = 0; i < n; ++i)
    if (x == set[i]) return true;
  return false;
}

// Validates a description; fills the internal shape.  `for_step` skips the
// chunk-related checks.
int check_desc(const tla_desc* d, tla::Shape* s, bool for_step) {
  if (!d) return fail(TLA_E_NULL, "desc is NULL");
  if (d->struct_size != (int32_t)sizeof(tla_desc))
    return fail(TLA_E_SHAPE, "desc->struct_size %d != %d", d->struct_size, (int)sizeof(tla_desc));
  if (d->variant != TLA_SGLA && d->variant != TLA_GDN)
    return fail(TLA_E_SHAPE, "variant %d is neither TLA_SGLA nor TLA_GDN", d->variant);
  if (d->in_dtype != TLA_F32 && d->in_dtype != TLA_BF16)
    return fail(TLA_E_SHAPE, "in_dtype %d", d->in_dtype);
  if (d->out_dtype != TLA_F32 && d->out_dtype != TLA_BF16)
    return fail(TLA_E_SHAPE, "out_dtype %d", d->out_dtype);
  if (d->B < 1 || d->H < 1) return fail(TLA_E_SHAPE, "B=%d H=%d must be >= 1", d->B, d->H);
  if (!for_step && d->T < 0) return fail(TLA_E_SHAPE, "T=%d must be >= 0", d->T);
  static const int Ks[] = {16, 32, 64, 128};
  static const int Es[] = {1, 2, 4, 8, 16, 32};
  static const int Cs[] = {16, 32, 64};
  if (!pow2_in(d->K, Ks, 4)) return fail(TLA_E_UNSUPPORTED, "K=%d not in {16,32,64,128}", d->K);
  if (d->V < 16 || d->V > 1024 || d->V % 16 != 0)
    return fail(TLA_E_UNSUPPORTED, "V=%d must be a multiple of 16 in [16, 1024]", d->V);
  if (!pow2_in(d->E, Es, 6)) return fail(TLA_E_UNSUPPORTED, "E=%d not in {1,2,4,8,16,32}", d->E);
  if (!for_step) {
    if (!pow2_in(d->chunk, Cs, 3)) return fail(TLA_E_UNSUPPORTED, "chunk=%d not in {16,32,64}", d->chunk);
    if (!tla::have_instance(d->K, d->chunk, d->E))
      return fail(TLA_E_UNSUPPORTED, "no kernel instance for K=%d chunk=%d E=%d", d->K, d->chunk, d->E);
    if (!tla::fits_lds(d->K, d->chunk, d->E, d->in_dtype == TLA_BF16) ||
        !tla::bwd_fits_lds(d->K, d->chunk, d->E, d->in_dtype == TLA_BF16))
      return fail(TLA_E_UNSUPPORTED, "K=%d chunk=%d E=%d with %s operands exceeds the LDS budget",
                  d->K, d->chunk, d->E, d->in_dtype == TLA_BF16 ? "bf16" : "fp32");
  } else {
    const bool ok = (d->K == 16 && d->E == 4) || (d->K == 32 && d->E == 4) ||
                    (d->K == 32 && d->E == 32) || (d->K == 64 && d->E == 8) ||
                    (d->K == 64 && d->E == 16) ||
                    (d->K == 128 && (d->E == 1 || d->E == 4 || d->E == 8 || d->E == 16));
    if (!ok) return fail(TLA_E_UNSUPPORTED, "no step instance for K=%d E=%d", d->K, d->E);
  }
  if ((double)d->B * d->H * (for_step ? 1 : (d->T > 0 ? d->T : 1)) * (d->K > d->V ? d->K : d->V) >
      (double)(1ull << 40))
    return fail(TLA_E_SHAPE, "problem too large");
  s->variant = d->variant;
  s->B = d->B;
  s->T = for_step ? 1 : d->T;
  s->H = d->H;
  s->K = d->K;
  s->V = d->V;
  s->E = d->E;
  s->C = for_step ? 16 : d->chunk;
  s->Nc = for_step ? 1 : (d->T + d->chunk - 1) / d->chunk;
  s->NH = d->B * d->H;
  s->in_bf16 = d->in_dtype == TLA_BF16;
  s->out_bf16 = d->out_dtype == TLA_BF16;
  s->has_beta = 0;
  s->cu = nullptr;
  s->total = 0;
  return TLA_OK;
}

// Packed variable-length batches: checks the host-side arguments and fills
// the packed fields of the shape (offsets stay on the device).
int check_varlen(const int32_t* cu_seqlens, long long total_tokens, tla::Shape* s) {
  if (!cu_seqlens) return fail(TLA_E_NULL, "cu_seqlens is NULL");
  if (((uintptr_t)cu_seqlens & 3u) != 0) return fail(TLA_E_ALIGN, "cu_seqlens is not 4-byte aligned");
  if (total_tokens < 0) return fail(TLA_E_SHAPE, "total_tokens=%lld must be >= 0", total_tokens);
  if (total_tokens > (long long)s->B * s->T)
    return fail(TLA_E_SHAPE, "total_tokens=%lld exceeds B * T = %lld (T is the longest sequence)",
                total_tokens, (long long)s->B * s->T);
  s->cu = cu_seqlens;
  s->total = total_tokens;
  return TLA_OK;
}

size_t esize(const tla::Shape& s) { return s.in_bf16 ? 2 : 4; }

// Buffer layouts.  The per-chunk prep results (coefficient vectors, gamma^C,
// M, Tu) live in the forward workspace for inference; a training forward
// writes them into `saved`, where the backward reads them again.
struct Layout {
  size_t p_coef, p_gC, p_ops, p_ninv, p_size;  // prep region, relative offsets
  size_t bwd_dS, bwd_dSlo, bwd_dU, bwd_dW, bwd_dqs, bwd_dks, bwd_dcoef, bwd_dgC, bwd_end;
  size_t sv_S, sv_U, sv_X, sv_prep, sv_end;
};

Layout layout(const tla::Shape& s) {
  Layout L;
  const size_t nch = (size_t)s.NH * s.Nc;
  const size_t es = esize(s);
  const size_t E4 = tla::round4(s.E);
  size_t o = 0;
  L.p_coef = o; o += align256(nch * 3 * s.E * s.C * 4);
  L.p_gC = o;   o += align256(nch * E4 * 4);
  L.p_ops = o;  o += align256(nch * tla::op_tile_bytes(s.K, s.C, s.in_bf16));
  L.p_ninv = o; o += s.variant == TLA_GDN ? align256(nch * s.C * s.C * 4) : 0;
  L.p_size = o;
  o = 0;
  L.bwd_dS = o;    o += align256(nch * s.E * s.K * s.V * es);
  L.bwd_dU = o;    o += align256(nch * s.C * s.V * 4);
  L.bwd_dW = o;    o += align256(nch * s.C * s.V * 4);
  L.bwd_dqs = o;   o += align256(nch * s.C * s.K * 4);
  L.bwd_dks = o;   o += align256(nch * s.C * s.K * 4);
  L.bwd_dcoef = o; o += align256(nch * 3 * s.E * s.C * 4);
  L.bwd_dgC = o;   o += align256(nch * E4 * 4);
  // low parts of the state gradients (bf16 operands, used when a final-state
  // gradient is given); last, so that a call without one needs only the
  // first bwd_dSlo bytes
  L.bwd_dSlo = o;  o += s.in_bf16 ? align256(nch * s.E * s.K * s.V * es) : 0;
  L.bwd_end = o;
  o = 0;
  L.sv_S = o;    o += align256(nch * s.E * s.K * s.V * es);
  L.sv_U = o;    o += align256(nch * s.C * s.V * 4);
  L.sv_X = o;    o += align256(nch * s.C * s.V * 4);
  L.sv_prep = o; o += L.p_size;
  L.sv_end = o;
  return L;
}

// `ninv`: a training forward's prep results, which also keep (I + L)^{-1}
// (GDN) and the transposed operand tiles for the backward
tla::PrepBufs prep_bufs(const Layout& L, const void* base, bool ninv) {
  char* b = (char*)base;
  return tla::PrepBufs{(float*)(b + L.p_coef), (float*)(b + L.p_gC), (void*)(b + L.p_ops),
                       (ninv && L.p_ninv < L.p_size) ? (float*)(b + L.p_ninv) : nullptr,
                       ninv ? 1 : 0};
}
tla::SavedBufs saved_bufs(const Layout& L, const void* saved) {
  char* b = (char*)saved;
  return tla::SavedBufs{b + L.sv_S, (float*)(b + L.sv_U), (float*)(b + L.sv_X)};
}

struct Range {
  const void* p;
  size_t n;
};
bool overlap(Range a, Range b) {
  if (!a.p || !b.p || !a.n || !b.n) return false;
  const char* a0 = (const char*)a.p;
  const char* b0 = (const char*)b.p;
  return a0 < b0 + b.n && b0 < a0 + a.n;
}

int device_fail(hipError_t e, const char* what) {
  return fail(TLA_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

// ------------------------------------------------------------- kernel timing
// Diagnostics only: while enabled, every kernel launch of the library is
// bracketed by a pair of HIP events recorded on the launch stream.  Events are
// pooled and reused; nothing is recorded when timing is off.
enum { PROF_PREP, PROF_FWD, PROF_BWD_REC, PROF_BWD_STATE, PROF_BWD_CHUNK, PROF_STEP,
       PROF_GATE_FWD, PROF_GATE_BWD, PROF_GATE_DW, PROF_HEADS_FWD, PROF_HEADS_BWD,
       PROF_CONV_FWD, PROF_CONV_BWD, PROF_PROJ_FWD, PROF_GEMM, PROF_TRANSPOSE, PROF_N };
const char* const kProfNames[PROF_N] = {"prep",         "fwd_recurrent",  "bwd_recurrent",
                                        "bwd_state",    "bwd_chunk",      "step",
                                        "out_gate_fwd", "out_gate_bwd",   "out_gate_dw",
                                        "gate_heads_fwd", "gate_heads_bwd", "conv_in_fwd",
                                        "conv_in_bwd", "proj_in_fwd", "proj_gemm", "transpose"};
struct ProfRec {
  int kind;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRec> g_prof;        // recorded launches since enable
std::vector<hipEvent_t> g_ev_pool;  // events available for reuse

hipEvent_t take_event() {
  if (!g_ev_pool.empty()) {
    hipEvent_t e = g_ev_pool.back();
    g_ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Launch wrapper: runs `launch` between two events when timing is enabled.
template <typename F>
hipError_t timed(int kind, hipStream_t st, F launch) {
  hipEvent_t a = nullptr, b = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (g_prof_on) {
      a = take_event();
      b = take_event();
    }
  }
  if (a && b) (void)hipEventRecord(a, st);
  hipError_t e = launch();
  if (a && b) {
    (void)hipEventRecord(b, st);
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof.push_back(ProfRec{kind, a, b});
  }
  return e;
}

}  // namespace

extern "C" {

int tla_version(void) { return TLA_VERSION; }

const char* tla_last_error(void) { return g_err; }

const char* tla_status_string(int st) {
  switch (st) {
    case TLA_OK: return "TLA_OK";
    case TLA_E_NULL: return "TLA_E_NULL: a required pointer is NULL";
    case TLA_E_SHAPE: return "TLA_E_SHAPE: a dimension is out of range";
    case TLA_E_UNSUPPORTED: return "TLA_E_UNSUPPORTED: no kernel instance for this shape";
    case TLA_E_ALIGN: return "TLA_E_ALIGN: a pointer is not 16-byte aligned";
    case TLA_E_WORKSPACE: return "TLA_E_WORKSPACE: workspace or saved buffer too small";
    case TLA_E_ALIAS: return "TLA_E_ALIAS: an output overlaps an input";
    case TLA_E_DEVICE: return "TLA_E_DEVICE: a HIP launch failed";
    default: return "unknown tla status";
  }
}

int tla_supported(const tla_desc* d) {
  tla::Shape s;
  return check_desc(d, &s, false) == TLA_OK ? 1 : 0;
}

size_t tla_workspace_bytes(const tla_desc* d, int op) {
  tla::Shape s;
  if (check_desc(d, &s, false) != TLA_OK) return 0;
  const Layout L = layout(s);
  if (op == TLA_OP_FWD) return L.p_ninv;  // an inference forward keeps no inverse
  if (op == TLA_OP_BWD) return L.bwd_end;
  return 0;
}

size_t tla_saved_bytes(const tla_desc* d) {
  tla::Shape s;
  if (check_desc(d, &s, false) != TLA_OK) return 0;
  return layout(s).sv_end;
}

static int fwd_impl(const tla_desc* d, const int32_t* cu, long long total, const void* q,
                    const void* k, const void* v, const void* q2, const void* k2, const float* g,
                    const float* beta, const float* s0, void* o, float* s_final, void* saved,
                    void* ws, size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  tla::Shape s;
  int rc = check_desc(d, &s, false);
  if (rc) return rc;
  if (cu && (rc = check_varlen(cu, total, &s))) return rc;
  const size_t ntok = (cu ? (size_t)total : (size_t)s.B * s.T) * s.H;
  if (ntok > 0 && (!q || !k || !v || !q2 || !k2 || !g || !o))
    return fail(TLA_E_NULL, "q, k, v, q2, k2, g and o are required");
  if (s.variant == TLA_GDN && ntok > 0 && !beta) return fail(TLA_E_NULL, "GDN needs beta");
  const void* ptrs[] = {q, k, v, q2, k2, g, beta, s0, o, s_final, saved, ws};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const Layout L = layout(s);
  const bool use_ws = ntok > 0 && !saved;  // a training forward keeps its prep results in saved
  if (use_ws && (!ws || ws_bytes < L.p_ninv))
    return fail(TLA_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, L.p_ninv);
  const size_t es = esize(s), os = s.out_bf16 ? 2 : 4;
  const size_t sbytes = (size_t)s.NH * s.E * s.K * s.V * 4;
  const Range ins[] = {{q, ntok * s.K * es}, {k, ntok * s.K * es}, {v, ntok * s.V * es},
                       {q2, ntok * s.E * es}, {k2, ntok * s.E * es}, {g, ntok * s.E * 4},
                       {beta, beta ? ntok * 4 : 0}, {s0, s0 ? sbytes : 0}};
  const Range outs[] = {{o, ntok * s.V * os}, {saved, saved ? L.sv_end : 0},
                        {ws, use_ws ? L.p_ninv : 0}};
  for (const Range& a : outs)
    for (const Range& b : ins)
      if (overlap(a, b)) return fail(TLA_E_ALIAS, "an output or buffer overlaps an input");
  if (s_final) {
    for (const Range& b : ins) {
      if (b.p == s0) continue;  // in place is allowed
      if (overlap({s_final, sbytes}, b)) return fail(TLA_E_ALIAS, "s_final overlaps an input");
    }
    if (s0 && s0 != s_final && overlap({s_final, sbytes}, {s0, sbytes}))
      return fail(TLA_E_ALIAS, "s_final partially overlaps s0");
    for (const Range& b : outs)
      if (overlap({s_final, sbytes}, b)) return fail(TLA_E_ALIAS, "s_final overlaps an output");
  }
  if (overlap(outs[0], outs[1]) || overlap(outs[0], outs[2]) || overlap(outs[1], outs[2]))
    return fail(TLA_E_ALIAS, "o, saved and ws must not overlap");

  hipStream_t st = (hipStream_t)stream;
  s.has_beta = beta != nullptr;
  tla::FwdIn in{q, k, v, q2, k2, g, beta, s0};
  const tla::PrepBufs pb =
      saved ? prep_bufs(L, (char*)saved + L.sv_prep, true) : prep_bufs(L, ws, false);
  hipError_t e;
  if (ntok > 0) {
    e = timed(PROF_PREP, st, [&] { return tla::launch_prep(s, in, pb, st); });
    if (e != hipSuccess) return device_fail(e, "prep kernel");
  }
  if (ntok > 0 || s_final) {
    tla::SavedBufs sv = saved_bufs(L, saved);
    e = timed(PROF_FWD, st, [&] {
      return tla::launch_fwd(s, in, pb, o, s_final, saved ? &sv : nullptr, st);
    });
    if (e != hipSuccess) return device_fail(e, "forward kernel");
  }
  return TLA_OK;
}

int tla_fwd(const tla_desc* d, const void* q, const void* k, const void* v, const void* q2,
            const void* k2, const float* g, const float* beta, const float* s0, void* o,
            float* s_final, void* saved, void* ws, size_t ws_bytes, void* stream) {
  return fwd_impl(d, nullptr, 0, q, k, v, q2, k2, g, beta, s0, o, s_final, saved, ws, ws_bytes,
                  stream);
}

// Device address of `scratch` on the current GPU, looked up once per device
// (with that device current) and kept.
static int scratch_ptr(void** out) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static void* ptrs[kMaxDev] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return device_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDev) return fail(TLA_E_DEVICE, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(mu);
  if (!ptrs[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return device_fail(e, "hipGetSymbolAddress(scratch)");
    ptrs[dev] = p;
  }
  *out = ptrs[dev];
  return TLA_OK;
}

int tla_fwd_noalloc(const tla_desc* d, const void* q, const void* k, const void* v,
                    const void* q2, const void* k2, const float* g, const float* beta,
                    const float* s0, void* o, float* s_final, void* stream) {
  g_err[0] = 0;
  tla::Shape s;
  int rc = check_desc(d, &s, false);
  if (rc) return rc;
  const size_t need = layout(s).p_ninv;  // the inference forward's workspace
  if (need > (size_t)TLA_NOALLOC_SCRATCH_BYTES)
    return fail(TLA_E_WORKSPACE,
                "tla_fwd_noalloc needs %zu bytes of scratch, above its maximum of %zu "
                "(use tla_fwd with a caller workspace)", need, (size_t)TLA_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((rc = scratch_ptr(&ws))) return rc;
  return fwd_impl(d, nullptr, 0, q, k, v, q2, k2, g, beta, s0, o, s_final, nullptr, ws,
                  (size_t)TLA_NOALLOC_SCRATCH_BYTES, stream);
}

int tla_fwd_varlen(const tla_desc* d, const int32_t* cu_seqlens, long long total_tokens,
                   const void* q, const void* k, const void* v, const void* q2, const void* k2,
                   const float* g, const float* beta, const float* s0, void* o, float* s_final,
                   void* saved, void* ws, size_t ws_bytes, void* stream) {
  if (!cu_seqlens) return fail(TLA_E_NULL, "cu_seqlens is NULL");
  return fwd_impl(d, cu_seqlens, total_tokens, q, k, v, q2, k2, g, beta, s0, o, s_final, saved,
                  ws, ws_bytes, stream);
}

static int bwd_impl(const tla_desc* d, const int32_t* cu, long long total, const void* q,
                    const void* k, const void* v, const void* q2, const void* k2, const float* g,
                    const float* beta, const float* s0, const void* dO, const float* dS_final,
                    const void* saved, void* dq, void* dk, void* dv, void* dq2, void* dk2,
                    float* dg, float* dbeta, float* ds0, void* ws, size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  tla::Shape s;
  int rc = check_desc(d, &s, false);
  if (rc) return rc;
  if (s.T < 1) return fail(TLA_E_SHAPE, "the backward needs T >= 1");
  if (cu && (rc = check_varlen(cu, total, &s))) return rc;
  if (s.V > 128) return fail(TLA_E_UNSUPPORTED, "the backward supports V <= 128 (V=%d)", s.V);
  const size_t ntok = (cu ? (size_t)total : (size_t)s.B * s.T) * s.H;
  if (!saved || !ws || (ntok > 0 && (!q || !k || !v || !q2 || !k2 || !g || !dO || !dq || !dk ||
                                     !dv || !dq2 || !dk2 || !dg)))
    return fail(TLA_E_NULL, "a required pointer is NULL");
  if (s.variant == TLA_GDN && ntok > 0 && !beta) return fail(TLA_E_NULL, "GDN needs beta");
  if ((beta == nullptr) != (dbeta == nullptr))
    return fail(TLA_E_NULL, "dbeta must be given exactly when beta is");
  const void* ptrs[] = {q, k, v, q2, k2, g, beta, s0, dO, dS_final, saved, dq,
                        dk, dv, dq2, dk2, dg, dbeta, ds0, ws};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const Layout L = layout(s);
  const bool pds = s.in_bf16 && dS_final;  // state gradients as bf16 (hi, lo) pairs
  const size_t ws_need = pds ? L.bwd_end : L.bwd_dSlo;
  if (ws_bytes < ws_need) return fail(TLA_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, ws_need);
  const size_t es = esize(s), os = s.out_bf16 ? 2 : 4;
  const size_t sbytes = (size_t)s.NH * s.E * s.K * s.V * 4;
  const Range ins[] = {{q, ntok * s.K * es}, {k, ntok * s.K * es}, {v, ntok * s.V * es},
                       {q2, ntok * s.E * es}, {k2, ntok * s.E * es}, {g, ntok * s.E * 4},
                       {beta, beta ? ntok * 4 : 0}, {s0, s0 ? sbytes : 0},
                       {dO, ntok * s.V * es}, {dS_final, dS_final ? sbytes : 0},
                       {saved, L.sv_end}};
  const Range outs[] = {{dq, ntok * s.K * os}, {dk, ntok * s.K * os}, {dv, ntok * s.V * os},
                        {dq2, ntok * s.E * os}, {dk2, ntok * s.E * os}, {dg, ntok * s.E * 4},
                        {dbeta, dbeta ? ntok * 4 : 0}, {ds0, ds0 ? sbytes : 0},
                        {ws, ws_need}};
  const int nouts = sizeof(outs) / sizeof(outs[0]);
  for (const Range& a : outs)
    for (const Range& b : ins)
      if (overlap(a, b)) return fail(TLA_E_ALIAS, "a gradient or the workspace overlaps an input");
  for (int i = 0; i < nouts; ++i)
    for (int j = i + 1; j < nouts; ++j)
      if (overlap(outs[i], outs[j])) return fail(TLA_E_ALIAS, "two outputs overlap");

  hipStream_t st = (hipStream_t)stream;
  s.has_beta = beta != nullptr;
  tla::FwdIn in{q, k, v, q2, k2, g, beta, s0};
  const tla::PrepBufs pb = prep_bufs(L, (const char*)saved + L.sv_prep, true);  // from the forward
  char* wb = (char*)ws;
  const tla::BwdBufs bb{wb + L.bwd_dS, pds ? wb + L.bwd_dSlo : nullptr,
                        (float*)(wb + L.bwd_dU), (float*)(wb + L.bwd_dW),
                        (float*)(wb + L.bwd_dqs), (float*)(wb + L.bwd_dks),
                        (float*)(wb + L.bwd_dcoef), (float*)(wb + L.bwd_dgC)};
  const tla::SavedBufs sv = saved_bufs(L, saved);
  hipError_t e = timed(PROF_BWD_REC, st,
            [&] { return tla::launch_bwd_rec(s, in, dO, dS_final, pb, bb, ds0, st); });
  if (e != hipSuccess) return device_fail(e, "backward recurrent kernel");
  e = timed(PROF_BWD_STATE, st, [&] { return tla::launch_bwd_state(s, in, dO, pb, sv, bb, st); });
  if (e != hipSuccess) return device_fail(e, "backward state-gradient kernel");
  e = timed(PROF_BWD_CHUNK, st, [&] {
    return tla::launch_bwd_chunk(s, in, dO, pb, sv, bb, dq, dk, dv, dq2, dk2, dg, dbeta, st);
  });
  if (e != hipSuccess) return device_fail(e, "backward chunk kernel");
  return TLA_OK;
}

int tla_bwd(const tla_desc* d, const void* q, const void* k, const void* v, const void* q2,
            const void* k2, const float* g, const float* beta, const float* s0, const void* dO,
            const float* dS_final, const void* saved, void* dq, void* dk, void* dv, void* dq2,
            void* dk2, float* dg, float* dbeta, float* ds0, void* ws, size_t ws_bytes,
            void* stream) {
  return bwd_impl(d, nullptr, 0, q, k, v, q2, k2, g, beta, s0, dO, dS_final, saved, dq, dk, dv,
                  dq2, dk2, dg, dbeta, ds0, ws, ws_bytes, stream);
}

int tla_bwd_varlen(const tla_desc* d, const int32_t* cu_seqlens, long long total_tokens,
                   const void* q, const void* k, const void* v, const void* q2, const void* k2,
                   const float* g, const float* beta, const float* s0, const void* dO,
                   const float* dS_final, const void* saved, void* dq, void* dk, void* dv,
                   void* dq2, void* dk2, float* dg, float* dbeta, float* ds0, void* ws,
                   size_t ws_bytes, void* stream) {
  if (!cu_seqlens) return fail(TLA_E_NULL, "cu_seqlens is NULL");
  return bwd_impl(d, cu_seqlens, total_tokens, q, k, v, q2, k2, g, beta, s0, dO, dS_final, saved,
                  dq, dk, dv, dq2, dk2, dg, dbeta, ds0, ws, ws_bytes, stream);
}

int tla_step(const tla_desc* d, const void* q, const void* k, const void* v, const void* q2,
             const void* k2, const float* g, const float* beta, float* state, void* o,
             void* stream) {
  g_err[0] = 0;
  tla::Shape s;
  int rc = check_desc(d, &s, true);
  if (rc) return rc;
  if (!q || !k || !v || !q2 || !k2 || !g || !state || !o)
    return fail(TLA_E_NULL, "q, k, v, q2, k2, g, state and o are required");
  if (s.variant == TLA_GDN && !beta) return fail(TLA_E_NULL, "GDN needs beta");
  const void* ptrs[] = {q, k, v, q2, k2, g, beta, state, o};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const size_t n = (size_t)s.NH, es = esize(s), os = s.out_bf16 ? 2 : 4;
  const Range ins[] = {{q, n * s.K * es}, {k, n * s.K * es}, {v, n * s.V * es},
                       {q2, n * s.E * es}, {k2, n * s.E * es}, {g, n * s.E * 4},
                       {beta, beta ? n * 4 : 0}};
  const Range outs[] = {{state, n * s.E * s.K * s.V * 4}, {o, n * s.V * os}};
  for (const Range& a : outs)
    for (const Range& b : ins)
      if (overlap(a, b)) return fail(TLA_E_ALIAS, "state or o overlaps an input");
  if (overlap(outs[0], outs[1])) return fail(TLA_E_ALIAS, "state and o overlap");
  s.has_beta = beta != nullptr;
  tla::FwdIn in{q, k, v, q2, k2, g, beta, nullptr};
  hipError_t e = timed(PROF_STEP, (hipStream_t)stream,
                       [&] { return tla::launch_step(s, in, state, o, (hipStream_t)stream); });
  if (e != hipSuccess) return device_fail(e, "step kernel");
  return TLA_OK;
}

// ------------------------------------------------------- output side of the mixer
static int gate_check(int dtype, long long rows, int V, float eps) {
  if (dtype != TLA_F32 && dtype != TLA_BF16) return fail(TLA_E_SHAPE, "dtype %d", dtype);
  if (rows < 0) return fail(TLA_E_SHAPE, "rows = %lld", rows);
  if (V != 16 && V != 32 && V != 64 && V != 128 && V != 256)
    return fail(TLA_E_UNSUPPORTED, "V = %d (16, 32, 64, 128 or 256)", V);
  if (!(eps >= 0.f) || eps > 3.4e38f) return fail(TLA_E_SHAPE, "eps must be finite and >= 0");
  return TLA_OK;
}

size_t tla_out_gate_workspace_bytes(long long rows, int V) {
  if (rows < 0 || V < 16 || V > 256 || (V & (V - 1))) return 0;
  return align256((size_t)tla::gate_blocks(rows, V) * V * sizeof(float));
}

int tla_out_gate_fwd(int dtype, long long rows, int V, const void* o, const void* z,
                     const float* w, float eps, void* y, void* stream) {
  g_err[0] = 0;
  int rc = gate_check(dtype, rows, V, eps);
  if (rc) return rc;
  if (!w || (rows > 0 && (!o || !z || !y))) return fail(TLA_E_NULL, "o, z, w and y are required");
  const void* ptrs[] = {o, z, w, y};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const size_t nb = (size_t)rows * V * (dtype == TLA_BF16 ? 2 : 4);
  const Range out{y, nb};
  if (overlap(out, {o, nb}) || overlap(out, {z, nb}) || overlap(out, {w, (size_t)V * 4}))
    return fail(TLA_E_ALIAS, "y overlaps an input");
  if (rows == 0) return TLA_OK;
  hipError_t e = timed(PROF_GATE_FWD, (hipStream_t)stream, [&] {
    return tla::launch_gate_fwd(dtype == TLA_BF16, rows, V, o, z, w, eps, y, (hipStream_t)stream);
  });
  if (e != hipSuccess) return device_fail(e, "output gate kernel");
  return TLA_OK;
}

int tla_out_gate_bwd(int dtype, long long rows, int V, const void* o, const void* z,
                     const float* w, float eps, const void* dy, void* d_o, void* dz, float* dw,
                     void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  int rc = gate_check(dtype, rows, V, eps);
  if (rc) return rc;
  if (!w || !dw || (rows > 0 && (!o || !z || !dy || !d_o || !dz)))
    return fail(TLA_E_NULL, "o, z, w, dy, d_o, dz and dw are required");
  const void* ptrs[] = {o, z, w, dy, d_o, dz, dw, workspace};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const size_t need = tla_out_gate_workspace_bytes(rows, V);
  if (!workspace || workspace_bytes < need)
    return fail(TLA_E_WORKSPACE, "workspace of %zu bytes needed", need);
  const size_t nb = (size_t)rows * V * (dtype == TLA_BF16 ? 2 : 4);
  const Range ins[] = {{o, nb}, {z, nb}, {w, (size_t)V * 4}, {dy, nb}};
  const Range outs[] = {{d_o, nb}, {dz, nb}, {dw, (size_t)V * 4}, {workspace, need}};
  for (const Range& a : outs)
    for (const Range& b : ins)
      if (overlap(a, b)) return fail(TLA_E_ALIAS, "an output or the workspace overlaps an input");
  for (int i = 0; i < 4; ++i)
    for (int j = i + 1; j < 4; ++j)
      if (overlap(outs[i], outs[j])) return fail(TLA_E_ALIAS, "two outputs overlap");
  hipStream_t st = (hipStream_t)stream;
  float* part = (float*)workspace;
  hipError_t e = timed(PROF_GATE_BWD, st, [&] {
    return tla::launch_gate_bwd(dtype == TLA_BF16, rows, V, o, z, w, eps, dy, d_o, dz, part, st);
  });
  if (e != hipSuccess) return device_fail(e, "output gate backward kernel");
  e = timed(PROF_GATE_DW, st, [&] { return tla::launch_gate_dw(rows, V, part, dw, st); });
  if (e != hipSuccess) return device_fail(e, "output gate dw kernel");
  return TLA_OK;
}

// ------------------------------------------------------------- gate heads
static int heads_check(int dtype, long long tokens, int H, int E) {
  if (dtype != TLA_F32 && dtype != TLA_BF16) return fail(TLA_E_SHAPE, "dtype %d", dtype);
  if (tokens < 0) return fail(TLA_E_SHAPE, "tokens = %lld", tokens);
  if (H < 1 || E < 1 || (long long)H * E > (1 << 20))
    return fail(TLA_E_SHAPE, "H = %d, E = %d (H, E >= 1, H * E <= 2^20)", H, E);
  return TLA_OK;
}

size_t tla_gate_heads_workspace_bytes(long long tokens, int H, int E) {
  if (tokens < 0 || H < 1 || E < 1 || (long long)H * E > (1 << 20)) return 0;
  return align256((size_t)tla::heads_map(tokens, H, E).nbg * 2 * H * E * sizeof(float));
}

int tla_gate_heads_fwd(int dtype, long long tokens, int H, int E, const void* x, const void* xb,
                       const float* A, const float* b, float* g, float* beta, void* stream) {
  g_err[0] = 0;
  int rc = heads_check(dtype, tokens, H, E);
  if (rc) return rc;
  if (!A || !b || (tokens > 0 && (!x || !g))) return fail(TLA_E_NULL, "x, A, b and g are required");
  if ((xb == nullptr) != (beta == nullptr)) return fail(TLA_E_NULL, "xb and beta go together");
  const void* ptrs[] = {x, xb, A, b, g, beta};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const size_t es = dtype == TLA_BF16 ? 2 : 4, nx = (size_t)tokens * H * E, nb = (size_t)tokens * H;
  const Range ins[] = {{x, nx * es}, {xb, xb ? nb * es : 0}, {A, (size_t)H * E * 4},
                       {b, (size_t)H * E * 4}};
  const Range outs[] = {{g, nx * 4}, {beta, beta ? nb * 4 : 0}};
  for (const Range& a : outs)
    for (const Range& c : ins)
      if (overlap(a, c)) return fail(TLA_E_ALIAS, "g or beta overlaps an input");
  if (overlap(outs[0], outs[1])) return fail(TLA_E_ALIAS, "g and beta overlap");
  if (tokens == 0) return TLA_OK;
  hipError_t e = timed(PROF_HEADS_FWD, (hipStream_t)stream, [&] {
    return tla::launch_heads_fwd(dtype == TLA_BF16, tokens, H, E, x, xb, A, b, g, beta,
                                 (hipStream_t)stream);
  });
  if (e != hipSuccess) return device_fail(e, "gate heads kernel");
  return TLA_OK;
}

int tla_gate_heads_bwd(int dtype, long long tokens, int H, int E, const void* x, const void* xb,
                       const float* A, const float* b, const float* dg, const float* dbeta,
                       void* dx, void* dxb, float* dA, float* db, void* workspace,
                       size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  int rc = heads_check(dtype, tokens, H, E);
  if (rc) return rc;
  if (!A || !b || !dA || !db || (tokens > 0 && (!x || !dg || !dx)))
    return fail(TLA_E_NULL, "x, A, b, dg, dx, dA and db are required");
  if ((xb == nullptr) != (dbeta == nullptr) || (xb == nullptr) != (dxb == nullptr))
    return fail(TLA_E_NULL, "xb, dbeta and dxb go together");
  const void* ptrs[] = {x, xb, A, b, dg, dbeta, dx, dxb, dA, db, workspace};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const size_t need = tla_gate_heads_workspace_bytes(tokens, H, E);
  if (!workspace || workspace_bytes < need)
    return fail(TLA_E_WORKSPACE, "workspace of %zu bytes needed", need);
  const size_t es = dtype == TLA_BF16 ? 2 : 4, nx = (size_t)tokens * H * E, nb = (size_t)tokens * H;
  const size_t np = (size_t)H * E * 4, nbb = xb ? nb : 0;
  const Range ins[] = {{x, nx * es}, {xb, nbb * es}, {A, np}, {b, np}, {dg, nx * 4}, {dbeta, nbb * 4}};
  const Range outs[] = {{dx, nx * es}, {dxb, nbb * es}, {dA, np}, {db, np}, {workspace, need}};
  for (const Range& a : outs)
    for (const Range& c : ins)
      if (overlap(a, c)) return fail(TLA_E_ALIAS, "an output or the workspace overlaps an input");
  for (int i = 0; i < 5; ++i)
    for (int j = i + 1; j < 5; ++j)
      if (overlap(outs[i], outs[j])) return fail(TLA_E_ALIAS, "two outputs overlap");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = timed(PROF_HEADS_BWD, st, [&] {
    return tla::launch_heads_bwd(dtype == TLA_BF16, tokens, H, E, x, xb, A, b, dg, dbeta, dx, dxb,
                                 dA, db, (float*)workspace, st);
  });
  if (e != hipSuccess) return device_fail(e, "gate heads backward kernel");
  return TLA_OK;
}

// ------------------------------------------------ input side of the mixer
static bool pow2_8_256(int x) { return x >= 8 && x <= 256 && (x & (x - 1)) == 0; }

static int conv_check(int dtype, int B, int T, int H, int K, int V, int E, int W, float eps) {
  if (dtype != TLA_F32 && dtype != TLA_BF16) return fail(TLA_E_SHAPE, "dtype %d", dtype);
  if (B < 0 || T < 0 || H < 1 || H > 1024) return fail(TLA_E_SHAPE, "B = %d, T = %d, H = %d", B, T, H);
  if (!pow2_8_256(K) || !pow2_8_256(E))
    return fail(TLA_E_UNSUPPORTED, "K = %d, E = %d (each one of 8, 16, ..., 256)", K, E);
  if (V < 8 || V > 1024 || V % 8) return fail(TLA_E_UNSUPPORTED, "V = %d (a multiple of 8 up to 1024)", V);
  if (W < 1 || W > 4) return fail(TLA_E_UNSUPPORTED, "W = %d (1 to 4 taps)", W);
  if ((H * (2 * K + V) / 8) % (E / 8))
    return fail(TLA_E_UNSUPPORTED, "H (2K + V) / 8 = %d is not a multiple of E / 8", H * (2 * K + V) / 8);
  if (!(eps >= 0.f) || eps > 3.4e38f) return fail(TLA_E_SHAPE, "eps must be finite and >= 0");
  if ((double)B * T * H * (2.0 * K + V + 2.0 * E) > 4e15) return fail(TLA_E_SHAPE, "problem too large");
  return TLA_OK;
}

size_t tla_conv_in_workspace_bytes(int B, int T, int H, int K, int V, int E, int W) {
  if (B < 0 || T < 0 || H < 1 || K < 1 || V < 1 || E < 1 || W < 1 || W > 4) return 0;
  const tla::ConvArgs a = tla::conv_args(B, T, H, K, V, E, W, 0.f, true);
  return align256((size_t)tla::conv_parts(a) * W * a.Ctot * sizeof(float));
}

int tla_conv_in_fwd(int dtype, int B, int T, int H, int K, int V, int E, int W, float eps,
                    const void* y, const float* w, void* q, void* k, void* v, void* q2, void* k2,
                    void* stream) {
  g_err[0] = 0;
  int rc = conv_check(dtype, B, T, H, K, V, E, W, eps);
  if (rc) return rc;
  const size_t n = (size_t)B * T * H, es = dtype == TLA_BF16 ? 2 : 4;
  if (!w || (n > 0 && (!y || !q || !k || !v || !q2 || !k2)))
    return fail(TLA_E_NULL, "y, w, q, k, v, q2 and k2 are required");
  const void* ptrs[] = {y, w, q, k, v, q2, k2};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const size_t C = (size_t)(2 * K + V + 2 * E);  // channels per token and head
  const Range ins[] = {{y, n * C * es}, {w, (size_t)W * H * C * 4}};
  const Range outs[] = {{q, n * K * es}, {k, n * K * es}, {v, n * V * es}, {q2, n * E * es},
                        {k2, n * E * es}};
  for (const Range& a : outs)
    for (const Range& b : ins)
      if (overlap(a, b)) return fail(TLA_E_ALIAS, "an output overlaps an input");
  for (int i = 0; i < 5; ++i)
    for (int j = i + 1; j < 5; ++j)
      if (overlap(outs[i], outs[j])) return fail(TLA_E_ALIAS, "two outputs overlap");
  if (n == 0) return TLA_OK;
  const tla::ConvArgs a = tla::conv_args(B, T, H, K, V, E, W, eps, false);
  void* const out[5] = {q, k, v, q2, k2};
  hipError_t e = timed(PROF_CONV_FWD, (hipStream_t)stream, [&] {
    return tla::launch_conv_fwd(dtype == TLA_BF16, a, y, w, out, (hipStream_t)stream);
  });
  if (e != hipSuccess) return device_fail(e, "input-side convolution kernel");
  return TLA_OK;
}

int tla_conv_in_bwd(int dtype, int B, int T, int H, int K, int V, int E, int W, float eps,
                    const void* y, const float* w, const void* dq, const void* dk, const void* dv,
                    const void* dq2, const void* dk2, void* dy, float* dw, void* workspace,
                    size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  int rc = conv_check(dtype, B, T, H, K, V, E, W, eps);
  if (rc) return rc;
  const size_t n = (size_t)B * T * H, es = dtype == TLA_BF16 ? 2 : 4;
  if (!w || !dw || (n > 0 && (!y || !dq || !dk || !dv || !dq2 || !dk2 || !dy)))
    return fail(TLA_E_NULL, "y, w, dq, dk, dv, dq2, dk2, dy and dw are required");
  const void* ptrs[] = {y, w, dq, dk, dv, dq2, dk2, dy, dw, workspace};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const size_t need = tla_conv_in_workspace_bytes(B, T, H, K, V, E, W);
  if (!workspace || workspace_bytes < need)
    return fail(TLA_E_WORKSPACE, "workspace of %zu bytes needed", need);
  const size_t C = (size_t)(2 * K + V + 2 * E);
  const Range ins[] = {{y, n * C * es},       {w, (size_t)W * H * C * 4}, {dq, n * K * es},
                       {dk, n * K * es},      {dv, n * V * es},           {dq2, n * E * es},
                       {dk2, n * E * es}};
  const Range outs[] = {{dy, n * C * es}, {dw, (size_t)W * H * C * 4}, {workspace, need}};
  for (const Range& a : outs)
    for (const Range& b : ins)
      if (overlap(a, b)) return fail(TLA_E_ALIAS, "an output or the workspace overlaps an input");
  for (int i = 0; i < 3; ++i)
    for (int j = i + 1; j < 3; ++j)
      if (overlap(outs[i], outs[j])) return fail(TLA_E_ALIAS, "two outputs overlap");
  const tla::ConvArgs a = tla::conv_args(B, T, H, K, V, E, W, eps, true);
  const void* const dout[5] = {dq, dk, dv, dq2, dk2};
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = timed(PROF_CONV_BWD, st, [&] {
    return tla::launch_conv_bwd(dtype == TLA_BF16, a, y, w, dout, dy, dw, (float*)workspace, st);
  });
  if (e != hipSuccess) return device_fail(e, "input-side convolution backward kernel");
  return TLA_OK;
}

// ------------------------------------------------ input projection (fused)
static int proj_check(int B, int T, int Dm, int H, int K, int V, int E, int W, float eps) {
  int rc = conv_check(TLA_BF16, B, T, H, K, V, E, W, eps);
  if (rc) return rc;
  if (K > 128 || E > 128)
    return fail(TLA_E_UNSUPPORTED, "K = %d, E = %d (each at most 128: a channel tile holds whole heads)", K, E);
  if (Dm < 8 || Dm > 65536 || Dm % 8)
    return fail(TLA_E_UNSUPPORTED, "Dm = %d (a multiple of 8 from 8 to 65536)", Dm);
  // row offsets within a tile are 32-bit: 256 rows of the longest contraction
  if ((double)B * T > 8.0e6) return fail(TLA_E_SHAPE, "B T = %.0f tokens (at most 8e6)", (double)B * T);
  return TLA_OK;
}

int tla_proj_in_fwd(int B, int T, int Dm, int H, int K, int V, int E, int W, float eps,
                    const void* u, const void* Wp, const float* w, void* q, void* k, void* v,
                    void* q2, void* k2, void* y, void* stream) {
  g_err[0] = 0;
  int rc = proj_check(B, T, Dm, H, K, V, E, W, eps);
  if (rc) return rc;
  const size_t n = (size_t)B * T, C = (size_t)H * (2 * K + V + 2 * E);
  if (!w || !Wp || (n > 0 && (!u || !q || !k || !v || !q2 || !k2)))
    return fail(TLA_E_NULL, "u, Wp, w, q, k, v, q2 and k2 are required");
  const void* ptrs[] = {u, Wp, w, q, k, v, q2, k2, y};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const Range ins[] = {{u, n * Dm * 2}, {Wp, C * Dm * 2}, {w, (size_t)W * C * 4}};
  const Range outs[] = {{q, n * H * K * 2}, {k, n * H * K * 2}, {v, n * H * V * 2},
                        {q2, n * H * E * 2}, {k2, n * H * E * 2}, {y, y ? n * C * 2 : 0}};
  for (const Range& a : outs)
    for (const Range& b : ins)
      if (overlap(a, b)) return fail(TLA_E_ALIAS, "an output overlaps an input");
  for (int i = 0; i < 6; ++i)
    for (int j = i + 1; j < 6; ++j)
      if (overlap(outs[i], outs[j])) return fail(TLA_E_ALIAS, "two outputs overlap");
  if (n == 0) return TLA_OK;
  const tla::ProjArgs a = tla::proj_args(B, T, Dm, H, K, V, E, W, eps);
  void* const out[5] = {q, k, v, q2, k2};
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = timed(PROF_PROJ_FWD, st, [&] { return tla::launch_proj_in(a, u, Wp, w, out, y, st); });
  if (e != hipSuccess) return device_fail(e, "input projection kernel");
  return TLA_OK;
}

// Workspace of the backward: dy [n][C], dy^T [C][n8], u^T [Dm][n8], Wp^T
// [Dm][C] (bf16; n8 = n rounded up to 8, the padding zero), the partial sums
// of the dWp GEMM's splits, and the convolution backward's partials.
struct ProjWs {
  size_t dy, dyT, uT, WpT, part, conv, end;
  int splits;
};
static ProjWs proj_ws(int B, int T, int Dm, int H, int K, int V, int E, int W) {
  ProjWs L;
  const size_t n = (size_t)B * T, n8 = (n + 7) / 8 * 8, C = (size_t)H * (2 * K + V + 2 * E);
  L.splits = tla::gemm_splits((long long)C, Dm, (long long)n8);
  size_t o = 0;
  L.dy = o;   o += align256(n * C * 2);
  L.dyT = o;  o += align256(C * n8 * 2);
  L.uT = o;   o += align256((size_t)Dm * n8 * 2);
  L.WpT = o;  o += align256((size_t)Dm * C * 2);
  L.part = o; o += L.splits > 1 ? align256((size_t)L.splits * C * Dm * 4) : 0;
  L.conv = o; o += tla_conv_in_workspace_bytes(B, T, H, K, V, E, W);
  L.end = o;
  return L;
}

size_t tla_proj_in_workspace_bytes(int B, int T, int Dm, int H, int K, int V, int E, int W) {
  if (B < 0 || T < 0 || Dm < 1 || H < 1 || K < 1 || V < 1 || E < 1 || W < 1 || W > 4) return 0;
  return proj_ws(B, T, Dm, H, K, V, E, W).end;
}

int tla_proj_in_bwd(int B, int T, int Dm, int H, int K, int V, int E, int W, float eps,
                    const void* u, const void* Wp, const float* w, const void* y, const void* dq,
                    const void* dk, const void* dv, const void* dq2, const void* dk2, void* du,
                    float* dWp, float* dw, void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  int rc = proj_check(B, T, Dm, H, K, V, E, W, eps);
  if (rc) return rc;
  const size_t n = (size_t)B * T, n8 = (n + 7) / 8 * 8, C = (size_t)H * (2 * K + V + 2 * E);
  if (!Wp || !w || !dWp || !dw || (n > 0 && (!u || !y || !dq || !dk || !dv || !dq2 || !dk2 || !du)))
    return fail(TLA_E_NULL, "u, Wp, w, y, dq, dk, dv, dq2, dk2, du, dWp and dw are required");
  const void* ptrs[] = {u, Wp, w, y, dq, dk, dv, dq2, dk2, du, dWp, dw, workspace};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", p);
  const ProjWs L = proj_ws(B, T, Dm, H, K, V, E, W);
  if (!workspace || workspace_bytes < L.end)
    return fail(TLA_E_WORKSPACE, "workspace of %zu bytes needed", L.end);
  const Range ins[] = {{u, n * Dm * 2},      {Wp, C * Dm * 2},     {w, (size_t)W * C * 4},
                       {y, n * C * 2},       {dq, n * H * K * 2},  {dk, n * H * K * 2},
                       {dv, n * H * V * 2},  {dq2, n * H * E * 2}, {dk2, n * H * E * 2}};
  const Range outs[] = {{du, n * Dm * 2}, {dWp, C * Dm * 4}, {dw, (size_t)W * C * 4},
                        {workspace, L.end}};
  for (const Range& a : outs)
    for (const Range& b : ins)
      if (overlap(a, b)) return fail(TLA_E_ALIAS, "an output or the workspace overlaps an input");
  for (int i = 0; i < 4; ++i)
    for (int j = i + 1; j < 4; ++j)
      if (overlap(outs[i], outs[j])) return fail(TLA_E_ALIAS, "two outputs overlap");
  char* ws = (char*)workspace;
  hipStream_t st = (hipStream_t)stream;
  const tla::ConvArgs ca = tla::conv_args(B, T, H, K, V, E, W, eps, true);
  const void* const dout[5] = {dq, dk, dv, dq2, dk2};
  void* dy = ws + L.dy;
  hipError_t e = timed(PROF_CONV_BWD, st, [&] {
    return tla::launch_conv_bwd(true, ca, y, w, dout, dy, dw, (float*)(ws + L.conv), st);
  });
  if (e != hipSuccess) return device_fail(e, "input-side convolution backward kernel");
  e = timed(PROF_TRANSPOSE, st, [&] {
    hipError_t r = tla::launch_transpose((long long)C, Dm, (long long)C, Wp, ws + L.WpT, st);
    if (r == hipSuccess) r = tla::launch_transpose((long long)n, (long long)C, (long long)n8, dy, ws + L.dyT, st);
    if (r == hipSuccess) r = tla::launch_transpose((long long)n, Dm, (long long)n8, u, ws + L.uT, st);
    return r;
  });
  if (e != hipSuccess) return device_fail(e, "transpose kernel");
  e = timed(PROF_GEMM, st, [&] {
    // du [n][Dm] = dy [n][C] (Wp^T [Dm][C])^T
    hipError_t r = tla::launch_gemm_nt((long long)n, Dm, (long long)C, dy, ws + L.WpT, du, true, Dm,
                                       1, nullptr, st);
    // dWp [C][Dm] = dy^T [C][n8] (u^T [Dm][n8])^T
    if (r == hipSuccess)
      r = tla::launch_gemm_nt((long long)C, Dm, (long long)n8, ws + L.dyT, ws + L.uT, dWp, false, Dm,
                              L.splits, (float*)(ws + L.part), st);
    return r;
  });
  if (e != hipSuccess) return device_fail(e, "projection gradient GEMM");
  return TLA_OK;
}

// ----------------------------------------------------------- diagnostics
size_t tla_mfma_rate_flop(int shape, int blocks, int iters) {
  if ((shape != 0 && shape != 1) || blocks < 1 || iters < 1) return 0;
  // per wave and round: 32 x 16x16x32 (16384 each) or 8 x 32x32x16 (32768 each)
  return (size_t)blocks * 4 * (size_t)iters * (shape == 0 ? 32 * 16384 : 8 * 32768);
}

int tla_mfma_rate(int shape, int blocks, int iters, float* sink, void* stream) {
  g_err[0] = 0;
  if (shape != 0 && shape != 1) return fail(TLA_E_SHAPE, "shape %d (0: 16x16x32, 1: 32x32x16)", shape);
  if (blocks < 1 || blocks > 65536 || iters < 1 || iters > (1 << 24))
    return fail(TLA_E_SHAPE, "blocks = %d, iters = %d", blocks, iters);
  if (!sink) return fail(TLA_E_NULL, "sink is required");
  if (misaligned(sink)) return fail(TLA_E_ALIGN, "pointer %p is not 16-byte aligned", (void*)sink);
  hipError_t e = tla::launch_mfma_rate(shape == 1, blocks, iters, sink, (hipStream_t)stream);
  if (e != hipSuccess) return device_fail(e, "MFMA rate kernel");
  return TLA_OK;
}

int tla_prof_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (ProfRec& r : g_prof) {
    g_ev_pool.push_back(r.a);
    g_ev_pool.push_back(r.b);
  }
  g_prof.clear();
  g_prof_on = on != 0;
  return TLA_OK;
}

int tla_prof_read(double* total_ms, int* launches, int n) {
  if (!total_ms || !launches || n < PROF_N) return fail(TLA_E_NULL, "tla_prof_read needs %d slots", PROF_N);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (int i = 0; i < n; ++i) {
    total_ms[i] = 0.0;
    launches[i] = 0;
  }
  for (const ProfRec& r : g_prof) {
    hipError_t e = hipEventSynchronize(r.b);
    if (e != hipSuccess) return device_fail(e, "event synchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return device_fail(e, "event elapsed time");
    total_ms[r.kind] += ms;
    launches[r.kind] += 1;
  }
  return TLA_OK;
}

const char* tla_prof_name(int i) { return (i >= 0 && i < PROF_N) ? kProfNames[i] : ""; }

}  // extern "C"
