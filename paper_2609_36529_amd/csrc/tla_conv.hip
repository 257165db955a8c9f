// The mixer's input side after the projection GEMM (section "Input
// projections", Alg. 2): one causal depthwise convolution over the channels
// of q, k, v, q' and k' of every head, SiLU on the q, k, v channels and
// softplus on the q', k' channels, then q, k, q', k' divided by their
// Euclidean norm (per token and head; x / sqrt(sum x^2 + eps)), v left as is.
// The outputs are the operator's q, k, v, q2, k2 in their [B][T][H][.] layouts.
//
// GEMM output y: [B][T][Ctot], Ctot = H (2K + V + 2E), channel blocks
// q | k | v | q' | k', each [H][width].  Taps w: [W][Ctot] fp32; the output at
// token t reads tokens t - W + 1 .. t of its own batch row (earlier tokens
// count as zero), tap j weighting token t - (W - 1) + j.
//
// HBM-bound.  A lane owns eight consecutive channels (one 16-byte access of
// bf16) and walks a run of consecutive tokens, keeping the last W - 1 inputs
// in registers, so every input is read once (plus a W - 1 token halo per
// run).  A head's K (or E) channels are K / 8 aligned lanes of one wave, whose
// sum of squares is a butterfly within that group.  Each wave of a workgroup
// takes its own run of the same channels.  The backward recomputes the
// forward per token, walks W - 1 tokens past its run to collect the taps'
// gradients of its last inputs, and reduces the tap gradient dw in a fixed
// order (per lane over its tokens, per workgroup over its four waves in wave
// order, then over the workgroups by a second kernel), so dw is bitwise
// reproducible.
#include <hip/hip_runtime.h>

#include "tla_common.hpp"
#include "tla_input_side.hpp"
#include "tla_internal.hpp"

namespace tla {

constexpr int CONV_NTHR = 256;  // four waves, one run of tokens each
constexpr int CONV_U = 2;       // forward: tokens per load batch (two batches in flight)

// Eight values of one token as loaded (packed bf16, or fp32), converted only
// where used: loads are unconditional from clamped addresses, so a batch of
// them stays in flight together (a load inside a lane-dependent branch would
// be waited for before the branch ends).
template <typename T> struct Tok8;
template <> struct Tok8<bf16_t> {
  uint4 a;
  __device__ __forceinline__ void ld(const bf16_t* p) { a = *(const uint4*)p; }
  __device__ __forceinline__ void cvt(float (&x)[8]) const {
    const bf16x8 b = __builtin_bit_cast(bf16x8, a);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = (float)b[i];
  }
};
template <> struct Tok8<float> {
  f32x4 a, b;
  __device__ __forceinline__ void ld(const float* p) {
    a = *(const f32x4*)p;
    b = *(const f32x4*)(p + 4);
  }
  __device__ __forceinline__ void cvt(float (&x)[8]) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[i] = a[i];
      x[4 + i] = b[i];
    }
  }
};

// raw loads of tokens t .. t + N - 1, clamped to tokens below `end` (end > 0);
// values of clamped tokens are never used
template <int N, typename T>
__device__ __forceinline__ void load_tokens(const T* p, size_t stride, int t, int end,
                                            Tok8<T> (&x)[N]) {
#pragma unroll
  for (int u = 0; u < N; ++u) x[u].ld(p + (size_t)min(t + u, end - 1) * stride);
}

// taps of the lane's channels and the W - 1 inputs before token t0 (zero
// before the row starts), all loads issued before any is used
template <int W, typename T>
__device__ __forceinline__ void load_prologue(const ConvArgs& a, const float* w, const T* yb, int cl,
                                              int t0, float (&wt)[W][8],
                                              float (&hist)[W > 1 ? W - 1 : 1][8]) {
  Tok8<float> rw[W];
  Tok8<T> rh[W > 1 ? W - 1 : 1];
#pragma unroll
  for (int j = 0; j < W; ++j) rw[j].ld(w + (size_t)j * a.Ctot + cl);
#pragma unroll
  for (int h = 0; h < W - 1; ++h) rh[h].ld(yb + (size_t)max(t0 - 1 - h, 0) * a.Ctot);
#pragma unroll
  for (int j = 0; j < W; ++j) rw[j].cvt(wt[j]);
#pragma unroll
  for (int h = 0; h < W - 1; ++h) {
    rh[h].cvt(hist[h]);
    if (t0 - 1 - h < 0)  // uniform over the wave
#pragma unroll
      for (int i = 0; i < 8; ++i) hist[h][i] = 0.f;
  }
}

// forward of tokens tt .. tt + CONV_U - 1 (those below t1)
template <int W, typename T>
__device__ __forceinline__ void fwd_batch(const ConvArgs& a, const ConvLane& L, bool on, bool silu,
                                          const float (&wt)[W][8],
                                          float (&hist)[W > 1 ? W - 1 : 1][8],
                                          const Tok8<T> (&xr)[CONV_U], int tt, int t1, T* out,
                                          size_t orow) {
#pragma unroll
  for (int u = 0; u < CONV_U; ++u) {
    if (tt + u >= t1) break;  // uniform over the wave
    float x[8], z[8], r[8], ss = 0.f;
    xr[u].cvt(x);
    conv8<W>(wt, hist, x, z);
    push_hist<W>(hist, x);
    act8(silu, z, r);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += r[i] * r[i];
    ss = lane_group_sum(ss, L.lpr);
    if (L.lpr) {
      const float inv = rsqrtf(ss + a.eps);
#pragma unroll
      for (int i = 0; i < 8; ++i) r[i] *= inv;
    }
    if (on) store8(out + (size_t)(tt + u) * orow, r);
  }
}

template <typename T, int W>
__global__ __launch_bounds__(CONV_NTHR) void k_conv_fwd(ConvArgs a, const T* __restrict__ y,
                                                        const float* __restrict__ w, T* q, T* k, T* v,
                                                        T* q2, T* k2) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = (blockIdx.y * 64 + lane) * 8;
  const bool on = c < a.Ctot;
  const long long run = (long long)blockIdx.x * 4 + wv;
  if (run >= (long long)a.B * a.runs_per_row) return;  // the whole wave
  const int b = (int)(run / a.runs_per_row);
  const int t0 = (int)(run % a.runs_per_row) * a.tb, t1 = min(t0 + a.tb, a.T);
  const int cl = on ? c : a.Ctot - 8;  // lanes past the channels read (and never use) the last ones
  const ConvLane L = conv_lane(a, cl);  // and take the last kind (never stored)
  const bool silu = L.kind < 3;
  T* out = pick(L.kind, q, k, v, q2, k2) + (size_t)b * a.T * a.H * L.width + L.off;
  const size_t orow = (size_t)a.H * L.width;
  const T* yb = y + (size_t)b * a.T * a.Ctot + cl;

  float wt[W][8], hist[W > 1 ? W - 1 : 1][8];  // hist[h] = y[t - 1 - h]
  load_prologue<W>(a, w, yb, cl, t0, wt, hist);
  // two batches in flight, used alternately: the loads of one batch are
  // issued before the other batch's stores, so waiting for them never waits
  // for stores as well
  Tok8<T> xa[CONV_U], xb[CONV_U];
  load_tokens<CONV_U>(yb, a.Ctot, t0, t1, xa);
  for (int tt = t0; tt < t1; tt += 2 * CONV_U) {
    load_tokens<CONV_U>(yb, a.Ctot, tt + CONV_U, t1, xb);
    fwd_batch<W>(a, L, on, silu, wt, hist, xa, tt, t1, out, orow);
    load_tokens<CONV_U>(yb, a.Ctot, tt + 2 * CONV_U, t1, xa);
    fwd_batch<W>(a, L, on, silu, wt, hist, xb, tt + CONV_U, t1, out, orow);
  }
}

constexpr int CONV_UB = 2;  // backward: tokens per load batch (two batches in flight)

// Backward state of one lane walking its run.
template <int W>
struct BwdLane {
  float wt[W][8];
  float hist[W > 1 ? W - 1 : 1][8];  // y[t - 1 - h]
  float dzh[W][8];                   // dz[t - j]
  float acc[W][8];                   // tap-gradient sums over the run's own tokens
};

// backward of tokens tt .. tt + CONV_UB - 1 (those below te): recompute the
// forward, dz through the norm and the activation, the taps' gradients, and
// dy of the token W - 1 places back
template <int W, typename T>
__device__ __forceinline__ void bwd_batch(const ConvArgs& a, const ConvLane& L, bool on, bool silu,
                                          BwdLane<W>& s, const Tok8<T> (&xr)[CONV_UB],
                                          const Tok8<T> (&gr)[CONV_UB], int tt, int t0, int t1,
                                          int te, T* dyb) {
#pragma unroll
  for (int u = 0; u < CONV_UB; ++u) {
    const int t = tt + u;
    if (t >= te) break;  // uniform over the wave
    float dz[8];
    if (t < a.T) {  // uniform
      float x[8], g[8], z[8], r[8], sl[8], ss = 0.f, sd = 0.f;
      xr[u].cvt(x);
      gr[u].cvt(g);
      conv8<W>(s.wt, s.hist, x, z);
      act8_slope(silu, z, r, sl);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ss += r[i] * r[i];
        sd += g[i] * r[i];
      }
      ss = lane_group_sum(ss, L.lpr);
      sd = lane_group_sum(sd, L.lpr);
      // n = r / rho, rho = sqrt(ss + eps):  dr = dn / rho - r <dn, r> / rho^3
      const float inv = L.lpr ? rsqrtf(ss + a.eps) : 1.f;
      const float cr = L.lpr ? sd * inv * inv * inv : 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) dz[i] = (g[i] * inv - r[i] * cr) * sl[i];
      if (t < t1) {  // the run's own tokens carry the tap gradient
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          s.acc[W - 1][i] += dz[i] * x[i];
#pragma unroll
          for (int h = 0; h < W - 1; ++h) s.acc[W - 2 - h][i] += dz[i] * s.hist[h][i];
        }
      }
      push_hist<W>(s.hist, x);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) dz[i] = 0.f;
    }
#pragma unroll
    for (int h = W - 1; h > 0; --h)
#pragma unroll
      for (int i = 0; i < 8; ++i) s.dzh[h][i] = s.dzh[h - 1][i];
#pragma unroll
    for (int i = 0; i < 8; ++i) s.dzh[0][i] = dz[i];
    // dy[t'] = sum_j w[j] dz[t' + W - 1 - j] for t' = t - (W - 1)
    const int tp = t - (W - 1);
    if (on && tp >= t0) {
      float o[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        o[i] = 0.f;
#pragma unroll
        for (int j = 0; j < W; ++j) o[i] += s.wt[j][i] * s.dzh[j][i];
      }
      store8(dyb + (size_t)tp * a.Ctot, o);
    }
  }
}

template <typename T, int W>
__global__ __launch_bounds__(CONV_NTHR) void k_conv_bwd(ConvArgs a, const T* __restrict__ y,
                                                        const float* __restrict__ w, const T* dq,
                                                        const T* dk, const T* dv, const T* dq2,
                                                        const T* dk2, T* __restrict__ dy,
                                                        float* __restrict__ part) {
  __shared__ float xch[3][W][8][64];  // waves 1..3 hand their dw sums to wave 0
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = (blockIdx.y * 64 + lane) * 8;
  const bool on = c < a.Ctot;
  const int cl = on ? c : a.Ctot - 8;  // lanes past the channels read (and never use) the last ones
  const long long run = (long long)blockIdx.x * 4 + wv;
  const bool live = run < (long long)a.B * a.runs_per_row;  // uniform over the wave
  BwdLane<W> s;
#pragma unroll
  for (int j = 0; j < W; ++j)
#pragma unroll
    for (int i = 0; i < 8; ++i) s.acc[j][i] = s.dzh[j][i] = 0.f;
  if (live) {
    const int b = (int)(run / a.runs_per_row);
    const int t0 = (int)(run % a.runs_per_row) * a.tb, t1 = min(t0 + a.tb, a.T);
    const int te = t1 + W - 1;    // dz is needed up to t1 + W - 2
    const int tl = min(te, a.T);  // of which these exist
    const ConvLane L = conv_lane(a, cl);
    const bool silu = L.kind < 3;
    const size_t orow = (size_t)a.H * L.width;
    const T* yb = y + (size_t)b * a.T * a.Ctot + cl;
    const T* db = pick(L.kind, dq, dk, dv, dq2, dk2) + (size_t)b * a.T * orow + L.off;
    T* dyb = dy + (size_t)b * a.T * a.Ctot + c;
    load_prologue<W>(a, w, yb, cl, t0, s.wt, s.hist);
    if (!on)
#pragma unroll
      for (int j = 0; j < W; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) s.wt[j][i] = 0.f;
    Tok8<T> xa[CONV_UB], ga[CONV_UB], xb[CONV_UB], gb[CONV_UB];
    load_tokens<CONV_UB>(yb, a.Ctot, t0, tl, xa);
    load_tokens<CONV_UB>(db, orow, t0, tl, ga);
    for (int tt = t0; tt < te; tt += 2 * CONV_UB) {
      load_tokens<CONV_UB>(yb, a.Ctot, tt + CONV_UB, tl, xb);
      load_tokens<CONV_UB>(db, orow, tt + CONV_UB, tl, gb);
      bwd_batch<W>(a, L, on, silu, s, xa, ga, tt, t0, t1, te, dyb);
      load_tokens<CONV_UB>(yb, a.Ctot, tt + 2 * CONV_UB, tl, xa);
      load_tokens<CONV_UB>(db, orow, tt + 2 * CONV_UB, tl, ga);
      bwd_batch<W>(a, L, on, silu, s, xb, gb, tt + CONV_UB, t0, t1, te, dyb);
    }
  }
  // dw partials: waves in order 0, 1, 2, 3
  if (wv > 0)
#pragma unroll
    for (int j = 0; j < W; ++j)
#pragma unroll
      for (int i = 0; i < 8; ++i) xch[wv - 1][j][i][lane] = s.acc[j][i];
  __syncthreads();
  if (wv == 0 && on) {
#pragma unroll
    for (int j = 0; j < W; ++j) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int q = 0; q < 3; ++q) s.acc[j][i] += xch[q][j][i][lane];
      store8(part + ((size_t)blockIdx.x * W + j) * a.Ctot + c, s.acc[j]);
    }
  }
}

// dw[n] = sum over the workgroups' partials in workgroup order: wave g of a
// workgroup sums partials g, g + 4, ... of 64 consecutive entries, then wave
// 0 adds the four sums in wave order.
__global__ __launch_bounds__(CONV_NTHR) void k_conv_dw(int nparts, int n, const float* part,
                                                       float* dw) {
  __shared__ float xch[3][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (col < n) {
    int p = wv;
    for (; p + 12 < nparts; p += 16) {  // four loads in flight
      const float v0 = part[(size_t)p * n + col], v1 = part[(size_t)(p + 4) * n + col];
      const float v2 = part[(size_t)(p + 8) * n + col], v3 = part[(size_t)(p + 12) * n + col];
      s += v0;
      s += v1;
      s += v2;
      s += v3;
    }
    for (; p < nparts; p += 4) s += part[(size_t)p * n + col];
  }
  if (wv > 0) xch[wv - 1][lane] = s;
  __syncthreads();
  if (wv == 0 && col < n) dw[col] = s + xch[0][lane] + xch[1][lane] + xch[2][lane];
}

ConvArgs conv_args(int B, int T, int H, int K, int V, int E, int W, float eps, bool backward) {
  ConvArgs a;
  a.B = B, a.T = T, a.H = H, a.K = K, a.V = V, a.E = E, a.W = W;
  a.Ctot = H * (2 * K + V + 2 * E);
  // shorter runs give more waves; the backward's runs stay longer since each
  // workgroup of runs adds a set of tap-gradient partials
  a.tb = backward ? 32 : 16;
  a.runs_per_row = T > 0 ? (T + a.tb - 1) / a.tb : 0;
  a.eps = eps;
  return a;
}

long long conv_parts(const ConvArgs& a) { return ((long long)a.B * a.runs_per_row + 3) / 4; }

template <typename T>
static hipError_t conv_fwd_t(const ConvArgs& a, const void* y, const float* w, void* const* out,
                             hipStream_t st) {
  const dim3 grid((unsigned)conv_parts(a), (unsigned)((a.Ctot / 8 + 63) / 64));
#define CONV_F(W_)                                                                                  \
  case W_:                                                                                          \
    hipLaunchKernelGGL((k_conv_fwd<T, W_>), grid, dim3(CONV_NTHR), 0, st, a, (const T*)y, w,        \
                       (T*)out[0], (T*)out[1], (T*)out[2], (T*)out[3], (T*)out[4]);                 \
    break;
  switch (a.W) {
    CONV_F(1) CONV_F(2) CONV_F(3) CONV_F(4)
    default: return hipErrorInvalidValue;
  }
#undef CONV_F
  return hipGetLastError();
}

template <typename T>
static hipError_t conv_bwd_t(const ConvArgs& a, const void* y, const float* w,
                             const void* const* dout, void* dy, float* part, hipStream_t st) {
  const dim3 grid((unsigned)conv_parts(a), (unsigned)((a.Ctot / 8 + 63) / 64));
#define CONV_B(W_)                                                                                  \
  case W_:                                                                                          \
    hipLaunchKernelGGL((k_conv_bwd<T, W_>), grid, dim3(CONV_NTHR), 0, st, a, (const T*)y, w,        \
                       (const T*)dout[0], (const T*)dout[1], (const T*)dout[2], (const T*)dout[3],  \
                       (const T*)dout[4], (T*)dy, part);                                            \
    break;
  switch (a.W) {
    CONV_B(1) CONV_B(2) CONV_B(3) CONV_B(4)
    default: return hipErrorInvalidValue;
  }
#undef CONV_B
  return hipGetLastError();
}

hipError_t launch_conv_fwd(bool bf16, const ConvArgs& a, const void* y, const float* w,
                           void* const* out, hipStream_t st) {
  return bf16 ? conv_fwd_t<bf16_t>(a, y, w, out, st) : conv_fwd_t<float>(a, y, w, out, st);
}

hipError_t launch_conv_bwd(bool bf16, const ConvArgs& a, const void* y, const float* w,
                           const void* const* dout, void* dy, float* dw, float* part,
                           hipStream_t st) {
  if (conv_parts(a) > 0) {
    hipError_t e = bf16 ? conv_bwd_t<bf16_t>(a, y, w, dout, dy, part, st)
                        : conv_bwd_t<float>(a, y, w, dout, dy, part, st);
    if (e != hipSuccess) return e;
  }
  const int n = a.W * a.Ctot;
  hipLaunchKernelGGL(k_conv_dw, dim3((n + 63) / 64), dim3(CONV_NTHR), 0, st, (int)conv_parts(a), n,
                     part, dw);
  return hipGetLastError();
}

}  // namespace tla
