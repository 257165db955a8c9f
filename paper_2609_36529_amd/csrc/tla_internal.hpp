// Internal interface between the C-ABI host code and the kernel files.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tla {

// Shapes and derived sizes shared by every launch of one call.
struct Shape {
  int variant;   // 0 sGLA, 1 GDN
  int B, T, H, K, V, E, C;
  int Nc;        // number of chunks = ceil(T / C)
  int NH;        // B * H
  int in_bf16;   // operand type of q, k, v, q2, k2, dO and gradients
  int out_bf16;  // type of o
  int has_beta;
  // Packed variable-length sequences: with cu != nullptr, sequence b is
  // tokens [cu[b], cu[b + 1]) of one packed batch of `total` tokens, T is
  // the longest length (it sizes the per-chunk buffers) and B the number
  // of sequences.  cu is a device array of B + 1 offsets.
  const int* cu;
  long long total;
};

// First token and length of sequence b.  Packed offsets are clamped to the
// packed batch and lengths to [0, T], so malformed offsets give wrong
// results but never address memory outside the tensors.
__device__ __forceinline__ size_t seq_begin(const Shape& s, int b) {
  if (!s.cu) return (size_t)b * s.T;
  const long long x = s.cu[b];
  return (size_t)(x < 0 ? 0 : (x > s.total ? s.total : x));
}
__device__ __forceinline__ int seq_len(const Shape& s, int b) {
  if (!s.cu) return s.T;
  const long long b0 = (long long)seq_begin(s, b);
  long long e = s.cu[b + 1];
  e = e > s.total ? s.total : e;
  const long long n = e - b0;
  return (int)(n < 0 ? 0 : (n > s.T ? s.T : n));
}

// Per-chunk quantities written by the prep kernel.  All arrays are indexed by
// ch = (b * H + h) * Nc + chunk.
struct PrepBufs {
  float* coef;   // [ch][3][E][C]  a = k2*gamma, b = q2*gamma, c = k2*gamma^C/gamma
  float* gC;     // [ch][E4]       gamma^C (E4 = E rounded up to 4)
  void* ops;     // [ch][op_tile_elems] operand tiles, see OpTiles
  float* ninv;   // [ch][C][C]     (I + L)^{-1} in fp32 (GDN training forward), or NULL
  int bwd_tiles; // training forward: also write Q^T (read only by the backward)
};

// Operand tiles of one chunk, in the operand type T and in the layouts the
// recurrent kernels copy into shared memory: M = (Q K^T) o R' (lower incl.
// diagonal) and Tu = (I + L)^{-1} diag(beta) (GDN), row-major, as bf16
// (hi, lo) pairs for bf16 operands (one fp32 copy for fp32 operands), then
// K^T and Q^T of the chunk (rows past T are zero; key k in row row_of_key(k),
// the key order of the recurrent kernels' state tiles).  Q^T serves the
// backward only: an inference forward leaves it unwritten.  (The backward
// reads M and Tu by columns for its M^T and Tu^T operands.)
// Element offsets within a chunk's block; part p (0 = hi, 1 = lo) of a
// matrix X starts at X + p * MAT.
template <typename T, int KD, int C>
struct OpTiles {
  static constexpr int NS = sizeof(T) == 2 ? 2 : 1;
  static constexpr size_t MAT = (size_t)C * C;
  static constexpr size_t M = 0, Tu = NS * MAT;
  static constexpr size_t Kt = 2 * NS * MAT, Qt = Kt + (size_t)KD * C;
  static constexpr size_t STRIDE = Qt + (size_t)KD * C;
};
// Bytes of one chunk's operand tiles (host side).
inline size_t op_tile_bytes(int K, int C, bool bf16) {
  const size_t ns = bf16 ? 2 : 1, es = bf16 ? 2 : 4;
  return (2 * ns * (size_t)C * C + 2 * (size_t)K * C) * es;
}

// Buffers the training forward stores for the backward (opaque layout).
struct SavedBufs {
  void* Sck;     // [ch][E][V/16][K][16] chunk-start states, operand type; row i of a
                 // tile holds key key_of_row(i), the recurrent kernels' register order
  float* U;      // [ch][C][V] delta-corrected values U
  float* X;      // [ch][C][V] residual V - W (GDN)
};

struct BwdBufs {
  void* dSck;    // [ch][E][V/16][K][16] state gradients at chunk ends, operand type
                 // (rows in the same key order as Sck)
  void* dSck_lo; // bf16 operands with a final-state gradient: the low bf16 part of
                 // the same gradients (dSck holds the rounded high part); else NULL
  float* dU;     // [ch][C][V]
  float* dW;     // [ch][C][V]
  float* dqs;    // [ch][C][K] state contributions to dq
  float* dks;    // [ch][C][K] state contributions to dk
  float* dcoef;  // [ch][3][E][C] gradients of the coefficient vectors a, b, c
  float* dgC;    // [ch][E4] gradient of gamma^C
};

struct FwdIn {
  const void *q, *k, *v, *q2, *k2;
  const float *g, *beta, *s0;
};

inline int round4(int x) { return (x + 3) & ~3; }

// Kernel launchers (return hipGetLastError() after the launch).
hipError_t launch_prep(const Shape& s, const FwdIn& in, const PrepBufs& p, hipStream_t st);
hipError_t launch_fwd(const Shape& s, const FwdIn& in, const PrepBufs& p, void* o,
                      float* s_final, const SavedBufs* saved, hipStream_t st);
hipError_t launch_bwd_rec(const Shape& s, const FwdIn& in, const void* dO, const float* dS_final,
                          const PrepBufs& p, const BwdBufs& bb, float* ds0, hipStream_t st);
hipError_t launch_bwd_state(const Shape& s, const FwdIn& in, const void* dO, const PrepBufs& p,
                            const SavedBufs& sv, const BwdBufs& bb, hipStream_t st);
hipError_t launch_bwd_chunk(const Shape& s, const FwdIn& in, const void* dO, const PrepBufs& p,
                            const SavedBufs& sv,
                            const BwdBufs& bb, void* dq, void* dk, void* dv, void* dq2,
                            void* dk2, float* dg, float* dbeta, hipStream_t st);
hipError_t launch_step(const Shape& s, const FwdIn& in, float* state, void* o, hipStream_t st);
// The mixer's output side (RMSNorm times a sigmoid gate), rows of V values.
int gate_blocks(long long rows, int V);  // workgroups of the row kernels (dw partials)
hipError_t launch_gate_fwd(bool bf16, long long rows, int V, const void* o, const void* z,
                           const float* w, float eps, void* y, hipStream_t st);
hipError_t launch_gate_bwd(bool bf16, long long rows, int V, const void* o, const void* z,
                           const float* w, float eps, const void* dy, void* d_o, void* dz,
                           float* dw_part, hipStream_t st);
hipError_t launch_gate_dw(long long rows, int V, const float* dw_part, float* dw, hipStream_t st);
// The gate heads (log forget gate, write strength) from their pre-activations.
struct HeadsMap {
  int R, U;       // token rows side by side, runs per workgroup
  long long nbg;  // workgroups for g (= sets of dA, db partials)
  long long nbb;  // workgroups for beta
};
HeadsMap heads_map(long long tokens, int H, int E);
hipError_t launch_heads_fwd(bool bf16, long long tokens, int H, int E, const void* x, const void* xb,
                            const float* A, const float* b, float* g, float* beta, hipStream_t st);
hipError_t launch_heads_bwd(bool bf16, long long tokens, int H, int E, const void* x, const void* xb,
                            const float* A, const float* b, const float* dg, const float* dbeta,
                            void* dx, void* dxb, float* dA, float* db, float* part, hipStream_t st);
// The mixer's input side after the projection GEMM: causal depthwise
// convolution, SiLU / softplus, L2 normalisation.
struct ConvArgs {
  int B, T, H, K, V, E, W;
  int Ctot;          // H (2K + V + 2E) channels per token
  int tb;            // tokens per run (one wave walks one run)
  int runs_per_row;  // ceil(T / tb)
  float eps;
};
ConvArgs conv_args(int B, int T, int H, int K, int V, int E, int W, float eps, bool backward);
long long conv_parts(const ConvArgs& a);  // workgroups along the runs (= dw partial sets)
hipError_t launch_conv_fwd(bool bf16, const ConvArgs& a, const void* y, const float* w,
                           void* const* out, hipStream_t st);
hipError_t launch_conv_bwd(bool bf16, const ConvArgs& a, const void* y, const float* w,
                           const void* const* dout, void* dy, float* dw, float* part,
                           hipStream_t st);

// The input projection with its epilogue fused (GEMM u Wp^T, then the
// input side above), and the plain GEMMs and transposes of its backward.
struct ProjArgs {
  int B, T, Dm, H, K, V, E, W;
  int Ctot;            // H (2K + V + 2E) channels per token
  int tiles_per_row;   // token tiles per batch row, ceil(T / 256)
  int n_mt, n_ct;      // token tiles (B tiles_per_row) and channel tiles (ceil(Ctot / 128))
  float eps;
};
ProjArgs proj_args(int B, int T, int Dm, int H, int K, int V, int E, int W, float eps);
hipError_t launch_proj_in(const ProjArgs& a, const void* u, const void* Wp, const float* w,
                          void* const* out, void* y, hipStream_t st);
// C[M][N] = A[M][K] B[N][K]^T (bf16 operands, rows K elements apart, K a
// multiple of 8); C fp32 or bf16 with rows ldc apart.  With splits > 1 the
// contraction is cut into that many ranges whose fp32 partial products go to
// part ([splits][M][N]) and are then summed in split order into C.
int gemm_splits(long long M, long long N, long long K);
hipError_t launch_gemm_nt(long long M, long long N, long long K, const void* A, const void* Bm,
                          void* C, bool c_bf16, long long ldc, int splits, float* part,
                          hipStream_t st);
// out [C][Rp] = in [R][C]^T (bf16), rows R .. Rp - 1 of the result zero
hipError_t launch_transpose(long long R, long long C, long long Rp, const void* in, void* out,
                            hipStream_t st);

// Diagnostics: back-to-back bf16 MFMAs on register accumulators.
hipError_t launch_mfma_rate(bool wide, int blocks, int iters, float* sink, hipStream_t st);

// Which (K, C, E) combinations have kernel instances, and whether the
// forward/backward shared-memory plan of an instance fits 160 KiB.
bool have_instance(int K, int C, int E);
bool fits_lds(int K, int C, int E, bool bf16);
bool bwd_fits_lds(int K, int C, int E, bool bf16);

}  // namespace tla
