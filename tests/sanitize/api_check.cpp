// Test infrastructure: drives the C ABI's host-side validation of
// include/tla.h (tla_api.cpp) in a build with the address and
// undefined-behaviour sanitizers on the host code (tests/test_sanitize.py).
// Every call below is rejected on the host before anything touches a device
// (this runs without a GPU); the size queries run on valid descriptions.
#include <stdint.h>
#include <initializer_list>
#include <stdio.h>
#include <string.h>

#include "../../include/tla.h"

static int fails = 0;
#define EXPECT(cond)                                              \
  do {                                                            \
    if (!(cond)) {                                                \
      fprintf(stderr, "%s:%d: %s (last error: %s)\n", __FILE__,   \
              __LINE__, #cond, tla_last_error());                 \
      ++fails;                                                    \
    }                                                             \
  } while (0)

static tla_desc make(int variant, int B, int T, int H, int K, int V, int E, int C, int dt) {
  tla_desc d;
  memset(&d, 0, sizeof(d));
  d.struct_size = (int32_t)sizeof(tla_desc);
  d.variant = variant;
  d.B = B, d.T = T, d.H = H, d.K = K, d.V = V, d.E = E, d.chunk = C;
  d.in_dtype = dt, d.out_dtype = dt;
  return d;
}

int main() {
  void* const P = (void*)(uintptr_t)0x7f0000000000ull;  // aligned fake device address, never used
  void* const Q = (void*)(uintptr_t)0x7f0000000008ull;  // misaligned
  char* base = (char*)P;
  tla_desc ok = make(TLA_GDN, 4, 4096, 8, 128, 128, 8, 64, TLA_BF16);
  EXPECT(tla_supported(&ok) == 1);
  EXPECT(tla_workspace_bytes(&ok, TLA_OP_FWD) > 0);
  EXPECT(tla_workspace_bytes(&ok, TLA_OP_BWD) > tla_workspace_bytes(&ok, TLA_OP_FWD));
  EXPECT(tla_saved_bytes(&ok) > 0);
  for (int K : {16, 32, 64, 128})
    for (int E : {1, 2, 4, 8, 16, 32})
      for (int C : {16, 32, 64})
        for (int V : {16, 48, 128, 1024}) {
          tla_desc d = make(TLA_SGLA, 1, 100, 2, K, V, E, C, TLA_F32);
          (void)tla_supported(&d);
          (void)tla_workspace_bytes(&d, TLA_OP_BWD);
          (void)tla_saved_bytes(&d);
        }
  // malformed descriptions
  tla_desc bad = ok;
  bad.struct_size = 3;
  EXPECT(tla_fwd(&bad, P, P, P, P, P, (float*)P, (float*)P, 0, P, 0, 0, P, 1 << 30, 0) == TLA_E_SHAPE);
  EXPECT(tla_fwd(0, P, P, P, P, P, (float*)P, (float*)P, 0, P, 0, 0, P, 1 << 30, 0) == TLA_E_NULL);
  bad = ok, bad.K = 96;
  EXPECT(tla_fwd(&bad, P, P, P, P, P, (float*)P, (float*)P, 0, P, 0, 0, P, 1 << 30, 0) == TLA_E_UNSUPPORTED);
  bad = ok, bad.V = 20;
  EXPECT(tla_fwd(&bad, P, P, P, P, P, (float*)P, (float*)P, 0, P, 0, 0, P, 1 << 30, 0) == TLA_E_UNSUPPORTED);
  bad = ok, bad.B = 0;
  EXPECT(tla_fwd(&bad, P, P, P, P, P, (float*)P, (float*)P, 0, P, 0, 0, P, 1 << 30, 0) == TLA_E_SHAPE);
  bad = ok, bad.B = 1 << 20, bad.T = 1 << 20;
  EXPECT(tla_fwd(&bad, P, P, P, P, P, (float*)P, (float*)P, 0, P, 0, 0, P, 1 << 30, 0) == TLA_E_SHAPE);
  // pointers, alignment, workspace, aliasing
  EXPECT(tla_fwd(&ok, P, P, P, P, P, (float*)P, 0, 0, P, 0, 0, P, 1 << 30, 0) == TLA_E_NULL);
  EXPECT(tla_fwd(&ok, Q, P, P, P, P, (float*)P, (float*)P, 0, P, 0, 0, P, 1 << 30, 0) == TLA_E_ALIGN);
  const size_t tok = (size_t)4 * 4096 * 8;
  char* q = base;
  char* k = q + tok * 256;
  char* v = k + tok * 256;
  char* q2 = v + tok * 256;
  char* k2 = q2 + tok * 16;
  char* g = k2 + tok * 16;
  char* beta = g + tok * 32;
  char* o = beta + tok * 4 + 4096;
  char* ws = o + tok * 256;
  EXPECT(tla_fwd(&ok, q, k, v, q2, k2, (float*)g, (float*)beta, 0, o, 0, 0, ws, 16, 0) == TLA_E_WORKSPACE);
  EXPECT(tla_fwd(&ok, q, k, v, q2, k2, (float*)g, (float*)beta, 0, q, 0, 0, ws, (size_t)1 << 40, 0) ==
         TLA_E_ALIAS);
  EXPECT(tla_bwd(&ok, q, k, v, q2, k2, (float*)g, (float*)beta, 0, o, 0, 0, o, o, o, o, o, (float*)o, 0,
                 0, ws, 1 << 30, 0) == TLA_E_NULL);
  EXPECT(tla_bwd(&ok, q, k, v, q2, k2, (float*)g, (float*)beta, 0, o, 0, ws, o, o, o, o, o, (float*)o, 0,
                 0, ws, 1 << 30, 0) == TLA_E_NULL);  // dbeta missing with beta given
  EXPECT(tla_bwd(&ok, q, k, v, q2, k2, (float*)g, (float*)beta, 0, o, 0, ws, o, o, o, o, o, (float*)o,
                 (float*)o, 0, ws, 16, 0) == TLA_E_WORKSPACE);
  bad = ok, bad.V = 256;
  EXPECT(tla_bwd(&bad, q, k, v, q2, k2, (float*)g, (float*)beta, 0, o, 0, ws, o, o, o, o, o, (float*)o,
                 (float*)o, 0, ws, 16, 0) == TLA_E_UNSUPPORTED);
  EXPECT(tla_step(&ok, P, P, P, P, P, (float*)P, 0, (float*)P, P, 0) == TLA_E_NULL);
  tla_desc st = make(TLA_GDN, 256, 1, 16, 128, 128, 3, 64, TLA_BF16);
  EXPECT(tla_step(&st, P, P, P, P, P, (float*)P, (float*)P, (float*)P, P, 0) == TLA_E_UNSUPPORTED);
  EXPECT(tla_fwd_varlen(&ok, 0, 10, q, k, v, q2, k2, (float*)g, (float*)beta, 0, o, 0, 0, ws, 1 << 30, 0) ==
         TLA_E_NULL);
  EXPECT(tla_fwd_varlen(&ok, (const int32_t*)P, -1, q, k, v, q2, k2, (float*)g, (float*)beta, 0, o, 0, 0,
                        ws, 1 << 30, 0) == TLA_E_SHAPE);
  tla_desc big = make(TLA_GDN, 4, 4096, 8, 128, 128, 8, 64, TLA_BF16);
  EXPECT(tla_fwd_noalloc(&big, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0) == TLA_E_WORKSPACE);
  // the mixer's side ops
  EXPECT(tla_out_gate_fwd(TLA_BF16, 10, 48, P, P, (float*)P, 1e-6f, P, 0) == TLA_E_UNSUPPORTED);
  EXPECT(tla_out_gate_fwd(TLA_BF16, 10, 64, P, P, (float*)P, -1.f, P, 0) == TLA_E_SHAPE);
  EXPECT(tla_out_gate_bwd(TLA_F32, 10, 64, P, P, (float*)P, 1e-6f, P, P, P, (float*)P, P, 0, 0) ==
         TLA_E_WORKSPACE);
  EXPECT(tla_gate_heads_fwd(TLA_F32, 10, 0, 8, P, 0, (float*)P, (float*)P, (float*)P, 0, 0) == TLA_E_SHAPE);
  EXPECT(tla_gate_heads_bwd(TLA_F32, 10, 2, 8, P, P, (float*)P, (float*)P, (float*)P, 0, P, P, (float*)P,
                            (float*)P, P, 1 << 20, 0) == TLA_E_NULL);
  EXPECT(tla_conv_in_fwd(TLA_BF16, 1, 10, 2, 128, 128, 8, 5, 1e-6f, P, (float*)P, P, P, P, P, P, 0) ==
         TLA_E_UNSUPPORTED);
  EXPECT(tla_conv_in_bwd(TLA_BF16, 1, 10, 2, 128, 128, 8, 4, 1e-6f, P, (float*)P, P, P, P, P, P, P,
                         (float*)P, P, 0, 0) == TLA_E_WORKSPACE);
  (void)tla_out_gate_workspace_bytes(1 << 20, 128);
  (void)tla_gate_heads_workspace_bytes(1 << 20, 8, 8);
  (void)tla_conv_in_workspace_bytes(4, 4096, 8, 128, 128, 8, 4);
  EXPECT(tla_proj_in_fwd(1, 10, 100, 2, 128, 128, 8, 4, 1e-6f, P, P, (float*)P, P, P, P, P, P, 0, 0) ==
         TLA_E_UNSUPPORTED);
  EXPECT(tla_proj_in_fwd(1, 10, 128, 2, 128, 128, 8, 4, 1e-6f, P, P, (float*)P, P, P, Q, P, P, 0, 0) ==
         TLA_E_ALIGN);
  EXPECT(tla_proj_in_bwd(1, 10, 128, 2, 128, 128, 8, 4, 1e-6f, P, P, (float*)P, P, P, P, P, P, P, P,
                         (float*)P, (float*)P, P, 0, 0) == TLA_E_WORKSPACE);
  (void)tla_proj_in_workspace_bytes(4, 4096, 2048, 8, 128, 128, 8, 4);
  for (int i = -1; i < 9; ++i) (void)tla_status_string(i);
  printf(fails ? "api check: %d FAILED\n" : "api check: ok\n", fails);
  return fails != 0;
}
