// Device helpers of the mixer's input side (section "Input projections",
// Alg. 2), shared by the convolution kernels and the fused projection: which
// output a lane's eight channels belong to, the activations with their
// slopes, and sums over a lane group.
#pragma once
#include <hip/hip_runtime.h>

#include "tla_common.hpp"

namespace tla {

// The destination of a lane's eight channels: kind (0 q, 1 k, 2 v, 3 q', 4 k'),
// offset within that kind's [H][width] row, width, and the lanes of its norm
// group (0: not normalised).
struct ConvLane {
  int kind, off, width, lpr;
};

// (A: any argument block with fields H, K, V, E)
template <typename A>
__device__ __forceinline__ ConvLane conv_lane(const A& a, int c) {
  const int e0 = a.H * a.K, e1 = 2 * e0, e2 = e1 + a.H * a.V, e3 = e2 + a.H * a.E;
  if (c < e0) return {0, c, a.K, a.K / 8};
  if (c < e1) return {1, c - e0, a.K, a.K / 8};
  if (c < e2) return {2, c - e1, a.V, 0};
  if (c < e3) return {3, c - e2, a.E, a.E / 8};
  return {4, c - e3, a.E, a.E / 8};
}

// sum over the lpr aligned lanes of the caller's group (lpr 0 or a power of
// two dividing 64, the same for every lane of a group; every lane of the wave
// takes part in every exchange).  Within a 16-lane row the partial sums of 2,
// 4, 8 and 16 lanes come from DPP moves (no shared-memory round trip), and
// each lane keeps the one of its group's size; groups of 32 or 64 lanes,
// when the wave has any, add the cross-row exchanges.
__device__ __forceinline__ float lane_group_sum(float x, int lpr) {
  const float s2 = x + dpp_f<0xB1>(x);      // quad_perm [1,0,3,2]
  const float s4 = s2 + dpp_f<0x4E>(s2);    // quad_perm [2,3,0,1]
  const float s8 = s4 + dpp_f<0x141>(s4);   // row_half_mirror
  const float s16 = s8 + dpp_f<0x140>(s8);  // row_mirror
  float r = lpr >= 16 ? s16 : lpr >= 8 ? s8 : lpr >= 4 ? s4 : lpr >= 2 ? s2 : x;
  if (__builtin_amdgcn_ballot_w64(lpr >= 32)) {  // uniform over the wave
    const float s32 = s16 + __shfl_xor(s16, 16, 64);
    const float s64 = s32 + __shfl_xor(s32, 32, 64);
    r = lpr >= 64 ? s64 : lpr >= 32 ? s32 : r;
  }
  return r;
}

template <typename P>
__device__ __forceinline__ P pick(int kind, P p0, P p1, P p2, P p3, P p4) {
  return kind == 0 ? p0 : kind == 1 ? p1 : kind == 2 ? p2 : kind == 3 ? p3 : p4;
}

__device__ __forceinline__ float sig_rcp(float z) { return __builtin_amdgcn_rcpf(1.f + __expf(-z)); }

// softplus(y) = max(y, 0) + log1p(e), e = exp(-|y|) in (0, 1], with log1p by
// the compensated form log(u) e / (u - 1), u = 1 + e rounded (exact where
// u = 1): a few ulps, far cheaper than a general log1p.
__device__ __forceinline__ float softplus_c(float y) {
  const float e = __expf(-fabsf(y));
  const float u = 1.f + e;
  const float l = u == 1.f ? e : logf(u) * (e * __builtin_amdgcn_rcpf(u - 1.f));
  return fmaxf(y, 0.f) + l;
}

// Activation of a lane's eight channels (SiLU for kinds q, k, v, softplus for
// q', k'), and with it the slope.  The choice is made once per lane, so a wave
// runs only its own branch (waves mix the two only where the v and q' blocks
// meet).  SiLU' = s (1 + z (1 - s)), s = sigmoid(z); softplus' = sigmoid.
__device__ __forceinline__ void act8(bool silu, const float (&z)[8], float (&r)[8]) {
  if (silu) {
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = z[i] * sig_rcp(z[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = softplus_c(z[i]);
  }
}
__device__ __forceinline__ void act8_slope(bool silu, const float (&z)[8], float (&r)[8],
                                           float (&d)[8]) {
  if (silu) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float sg = sig_rcp(z[i]);
      r[i] = z[i] * sg;
      d[i] = sg * (1.f + z[i] * (1.f - sg));
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      r[i] = softplus_c(z[i]);
      d[i] = sig_rcp(z[i]);
    }
  }
}

// conv output of one token: taps over the history (hist[h] = y[t - 1 - h]) and y[t]
template <int W>
__device__ __forceinline__ void conv8(const float (&wt)[W][8], const float (&hist)[W > 1 ? W - 1 : 1][8],
                                      const float (&x)[8], float (&z)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    z[i] = wt[W - 1][i] * x[i];
#pragma unroll
    for (int h = 0; h < W - 1; ++h) z[i] += wt[W - 2 - h][i] * hist[h][i];
  }
}
template <int W>
__device__ __forceinline__ void push_hist(float (&hist)[W > 1 ? W - 1 : 1][8], const float (&x)[8]) {
#pragma unroll
  for (int h = W - 2; h > 0; --h)
#pragma unroll
    for (int i = 0; i < 8; ++i) hist[h][i] = hist[h - 1][i];
  if (W > 1)
#pragma unroll
    for (int i = 0; i < 8; ++i) hist[0][i] = x[i];
}

}  // namespace tla
