// The output side of the mixer (Alg. 2, the mixer's last line): per row of
// a head's V values,
//   y = o / sqrt(mean(o^2) + eps) * w * sigmoid(z),
// and its backward.  HBM-bound row kernels: V / 8 lanes per row, each lane
// holding eight consecutive values (one 16-byte access per bf16 operand),
// the mean square reduced within the row's lane group.  The gain gradient dw
// (a sum over all rows) is reduced in a fixed order: per lane over its rows
// (a fixed grid-stride set), per workgroup over its lanes, then over the
// workgroups by a second kernel, so it is bitwise reproducible.
#include <hip/hip_runtime.h>

#include "tla_common.hpp"
#include "tla_internal.hpp"

namespace tla {

constexpr int GATE_NTHR = 256;  // four waves

// sum over the LPR lanes of a row's group (aligned, a power of two)
template <int LPR>
__device__ __forceinline__ float group_sum(float x) {
#pragma unroll
  for (int m = 1; m < LPR; m <<= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// rows handled by one workgroup per grid-stride step
template <int V> constexpr int gate_rows_per_block() { return (GATE_NTHR / 64) * (64 / (V / 8)); }

template <typename T, int V>
__global__ __launch_bounds__(GATE_NTHR) void k_gate_fwd(long long rows, const T* o, const T* z,
                                                        const float* w, float eps, T* y) {
  constexpr int LPR = V / 8, RPW = 64 / LPR, RPB = gate_rows_per_block<V>();
  const int l = lane_id(), wv = threadIdx.x >> 6;
  const int c0 = 8 * (l % LPR);
  float wg[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) wg[i] = w[c0 + i];
  for (long long r0 = (long long)blockIdx.x * RPB; r0 < rows; r0 += (long long)gridDim.x * RPB) {
    const long long r = r0 + wv * RPW + l / LPR;
    const bool ok = r < rows;
    const size_t off = (size_t)(ok ? r : 0) * V + c0;
    float x[8], g[8];
    load8(o + off, x);
    load8(z + off, g);
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += x[i] * x[i];
    const float inv = 1.f / sqrtf(group_sum<LPR>(ss) / V + eps);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = x[i] * inv * wg[i] * sigmoidf_(g[i]);
    if (ok) store8(y + off, x);
  }
}

template <typename T, int V>
__global__ __launch_bounds__(GATE_NTHR) void k_gate_bwd(long long rows, const T* o, const T* z,
                                                        const float* w, float eps, const T* dy, T* d_o,
                                                        T* dz, float* dw_part) {
  constexpr int LPR = V / 8, RPW = 64 / LPR, RPB = gate_rows_per_block<V>();
  __shared__ float red[GATE_NTHR][8];
  const int l = lane_id(), wv = threadIdx.x >> 6;
  const int c0 = 8 * (l % LPR);
  float wg[8], dwp[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    wg[i] = w[c0 + i];
    dwp[i] = 0.f;
  }
  for (long long r0 = (long long)blockIdx.x * RPB; r0 < rows; r0 += (long long)gridDim.x * RPB) {
    const long long r = r0 + wv * RPW + l / LPR;
    const bool ok = r < rows;
    const size_t off = (size_t)(ok ? r : 0) * V + c0;
    float x[8], g[8], d[8];
    load8(o + off, x);
    load8(z + off, g);
    load8(dy + off, d);
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += x[i] * x[i];
    const float inv = 1.f / sqrtf(group_sum<LPR>(ss) / V + eps);
    float dn[8], nn[8], dzv[8], dot = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float s = sigmoidf_(g[i]);
      nn[i] = x[i] * inv;
      dzv[i] = d[i] * wg[i] * nn[i] * s * (1.f - s);
      dn[i] = d[i] * wg[i] * s;
      dot += dn[i] * nn[i];
      if (ok) dwp[i] += d[i] * nn[i] * s;
    }
    const float mdot = group_sum<LPR>(dot) / V;
    float dov[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) dov[i] = inv * (dn[i] - nn[i] * mdot);
    if (ok) {
      store8(d_o + off, dov);
      store8(dz + off, dzv);
    }
  }
  // workgroup partial of dw: column c sums, in a fixed order, the lanes that
  // hold it (lane l holds columns 8 (l % LPR) .. + 7 in every wave)
#pragma unroll
  for (int i = 0; i < 8; ++i) red[threadIdx.x][i] = dwp[i];
  __syncthreads();
  for (int c = threadIdx.x; c < V; c += GATE_NTHR) {
    float acc = 0.f;
    for (int t = c / 8; t < GATE_NTHR; t += LPR) acc += red[t][c % 8];
    dw_part[(size_t)blockIdx.x * V + c] = acc;
  }
}

// dw[c] = sum over the workgroups' partials (one workgroup per column c):
// thread t sums partials t, t + 256, ... in order, then a fixed binary tree
// over the threads (the same order on every call)
__global__ __launch_bounds__(GATE_NTHR) void k_gate_dw(int nblocks, int V, const float* dw_part,
                                                       float* dw) {
  __shared__ float red[GATE_NTHR];
  const int c = blockIdx.x, t = threadIdx.x;
  float acc = 0.f;
  for (int b = t; b < nblocks; b += GATE_NTHR) acc += dw_part[(size_t)b * V + c];
  red[t] = acc;
  __syncthreads();
#pragma unroll
  for (int m = GATE_NTHR / 2; m > 0; m >>= 1) {
    if (t < m) red[t] += red[t + m];
    __syncthreads();
  }
  if (t == 0) dw[c] = red[0];
}

// workgroups of the row kernels: enough to keep several per CU in flight;
// the backward's count is also the number of dw partials per column
static int gate_grid(long long rows, int V, long long cap) {
  const long long rpb = (GATE_NTHR / 64) * (64 / (V / 8));
  long long nb = (rows + rpb - 1) / rpb;
  if (nb > cap) nb = cap;
  return nb < 1 ? 1 : (int)nb;
}
int gate_blocks(long long rows, int V) { return gate_grid(rows, V, 1024); }

// ------------------------------------------------------------ gate heads
// Alg. 2's forget gate and write strength from their pre-activations:
//   g[n, h, e] = -exp(A[h, e]) softplus(x[n, h, e] + b[h, e])   (= log alpha <= 0)
//   beta[n, h] = sigmoid(xb[n, h])
// x is [tokens][HE] (HE = H * E columns).  Thread t of a g workgroup owns
// column c = t % HE and token row r = t / HE of each run of R = 256 / HE
// consecutive tokens (HE >= 256: R = 1, columns t, t + 256, ...); a workgroup
// covers U runs, R U tokens, and issues all U loads of a thread before any
// arithmetic.  The backward's per-column sums (dA, db) are therefore formed in
// a fixed order: each thread over its U tokens, then over the R rows of the
// workgroup, then one workgroup per column over the workgroups.  Workgroups
// past the g ones handle beta, HEAD_BPT consecutive (token, head) values per
// thread.
constexpr int HEAD_UMAX = 8;  // token runs per workgroup, at most
constexpr int HEAD_BPT = 4;   // beta values per thread


HeadsMap heads_map(long long tokens, int H, int E) {
  HeadsMap m;
  const long long HE = (long long)H * E;
  m.R = HE >= GATE_NTHR ? 1 : GATE_NTHR / (int)HE;
  m.U = HEAD_UMAX;  // fewer runs per workgroup while that leaves under 1024 workgroups
  while (m.U > 1 && (tokens + (long long)m.R * m.U - 1) / ((long long)m.R * m.U) < 1024) m.U /= 2;
  const long long nbg = (tokens + (long long)m.R * m.U - 1) / ((long long)m.R * m.U);
  m.nbg = nbg < 1 ? 1 : nbg;
  m.nbb = (tokens * H + GATE_NTHR * HEAD_BPT - 1) / (GATE_NTHR * HEAD_BPT);
  return m;
}

template <typename T>
__global__ __launch_bounds__(GATE_NTHR) void k_heads_fwd(long long tokens, int H, int HE, int R, int U,
                                                         int nbg, const T* x, const T* xb, const float* A,
                                                         const float* b, float* g, float* beta) {
  const int t = threadIdx.x;
  if ((int)blockIdx.x >= nbg) {  // write strength
    const long long NB = tokens * H;
    const long long j0 = ((long long)(blockIdx.x - nbg) * GATE_NTHR + t) * HEAD_BPT;
#pragma unroll
    for (int k = 0; k < HEAD_BPT; ++k)
      if (j0 + k < NB) beta[j0 + k] = sigmoidf_(Elem<T>::to_f(xb[j0 + k]));
    return;
  }
  const bool wide = HE >= GATE_NTHR;
  const int r = wide ? 0 : t / HE;
  if (r >= R) return;
  const long long n0 = (long long)blockIdx.x * R * U + r;
  for (int c = wide ? t : t % HE; c < HE; c += GATE_NTHR) {
    const float ea = __expf(A[c]), bc = b[c];
    float xv[HEAD_UMAX];
#pragma unroll
    for (int u = 0; u < HEAD_UMAX; ++u) {
      const long long n = n0 + (long long)u * R;
      xv[u] = (u < U && n < tokens) ? Elem<T>::to_f(x[n * HE + c]) : 0.f;
    }
#pragma unroll
    for (int u = 0; u < HEAD_UMAX; ++u) {
      const long long n = n0 + (long long)u * R;
      if (u < U && n < tokens) g[n * HE + c] = -ea * softplusf_(xv[u] + bc);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(GATE_NTHR) void k_heads_bwd(long long tokens, int H, int HE, int R, int U,
                                                         int nbg, const T* x, const T* xb, const float* A,
                                                         const float* b, const float* dg,
                                                         const float* dbeta, T* dx, T* dxb,
                                                         float* part) {
  const int t = threadIdx.x;
  if ((int)blockIdx.x >= nbg) {  // write strength: dxb = dbeta sigmoid'(xb)
    const long long NB = tokens * H;
    const long long j0 = ((long long)(blockIdx.x - nbg) * GATE_NTHR + t) * HEAD_BPT;
#pragma unroll
    for (int k = 0; k < HEAD_BPT; ++k)
      if (j0 + k < NB) {
        // beta (1 - beta) as sigmoid(x) sigmoid(-x): no cancellation once beta rounds to 1
        const float xv = Elem<T>::to_f(xb[j0 + k]);
        dxb[j0 + k] = Elem<T>::from_f(dbeta[j0 + k] * sigmoidf_(xv) * sigmoidf_(-xv));
      }
    return;
  }
  __shared__ float red[2][GATE_NTHR];
  const bool wide = HE >= GATE_NTHR;
  const int r = wide ? 0 : t / HE;
  const long long n0 = (long long)blockIdx.x * R * U + r;
  float* pa = part + (size_t)blockIdx.x * 2 * HE;  // this workgroup's partials of dA, then db
  for (int c = wide ? t : t % HE; c < HE; c += GATE_NTHR) {
    float sa = 0.f, sb = 0.f;
    if (r < R) {
      const float ea = __expf(A[c]), bc = b[c];
      float xv[HEAD_UMAX], dv[HEAD_UMAX];
#pragma unroll
      for (int u = 0; u < HEAD_UMAX; ++u) {
        const long long n = n0 + (long long)u * R;
        const bool ok = u < U && n < tokens;
        xv[u] = ok ? Elem<T>::to_f(x[n * HE + c]) : 0.f;
        dv[u] = ok ? dg[n * HE + c] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < HEAD_UMAX; ++u) {
        const long long n = n0 + (long long)u * R;
        if (u < U && n < tokens) {
          const float y = xv[u] + bc;
          const float dxx = -dv[u] * ea * sigmoidf_(y);
          dx[n * HE + c] = Elem<T>::from_f(dxx);
          sa += dv[u] * (-ea * softplusf_(y));
          sb += dxx;
        }
      }
    }
    if (wide) {  // one row: the thread's sums are the workgroup's
      pa[c] = sa;
      pa[HE + c] = sb;
    } else {  // sum the R rows of column c in row order
      red[0][t] = sa;
      red[1][t] = sb;
      __syncthreads();
      if (t < HE) {
        float a = 0.f, bb = 0.f;
        for (int q = 0; q < R; ++q) {
          a += red[0][q * HE + t];
          bb += red[1][q * HE + t];
        }
        pa[t] = a;
        pa[HE + t] = bb;
      }
    }
  }
}

// dA[c], db[c]: one workgroup per column, fixed-order sums of the partials
__global__ __launch_bounds__(GATE_NTHR) void k_heads_sum(int nblocks, int HE, const float* part,
                                                         float* dA, float* db) {
  __shared__ float red[2][GATE_NTHR];
  const int c = blockIdx.x, t = threadIdx.x;
  float a = 0.f, bb = 0.f;
  for (int k = t; k < nblocks; k += GATE_NTHR) {
    a += part[((size_t)k * 2 + 0) * HE + c];
    bb += part[((size_t)k * 2 + 1) * HE + c];
  }
  red[0][t] = a;
  red[1][t] = bb;
  __syncthreads();
#pragma unroll
  for (int m = GATE_NTHR / 2; m > 0; m >>= 1) {
    if (t < m) {
      red[0][t] += red[0][t + m];
      red[1][t] += red[1][t + m];
    }
    __syncthreads();
  }
  if (t == 0) {
    dA[c] = red[0][0];
    db[c] = red[1][0];
  }
}

hipError_t launch_heads_fwd(bool bf16, long long tokens, int H, int E, const void* x, const void* xb,
                            const float* A, const float* b, float* g, float* beta, hipStream_t st) {
  const HeadsMap m = heads_map(tokens, H, E);
  const long long nbb = xb ? m.nbb : 0;
  if (m.nbg + nbb > 0x7fffffffLL) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(m.nbg + nbb));
  if (bf16)
    hipLaunchKernelGGL(k_heads_fwd<bf16_t>, grid, dim3(GATE_NTHR), 0, st, tokens, H, H * E, m.R, m.U,
                       (int)m.nbg, (const bf16_t*)x, (const bf16_t*)xb, A, b, g, beta);
  else
    hipLaunchKernelGGL(k_heads_fwd<float>, grid, dim3(GATE_NTHR), 0, st, tokens, H, H * E, m.R, m.U,
                       (int)m.nbg, (const float*)x, (const float*)xb, A, b, g, beta);
  return hipGetLastError();
}

hipError_t launch_heads_bwd(bool bf16, long long tokens, int H, int E, const void* x, const void* xb,
                            const float* A, const float* b, const float* dg, const float* dbeta,
                            void* dx, void* dxb, float* dA, float* db, float* part, hipStream_t st) {
  const HeadsMap m = heads_map(tokens, H, E);
  const long long nbb = xb ? m.nbb : 0;
  if (m.nbg + nbb > 0x7fffffffLL) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(m.nbg + nbb));
  if (bf16)
    hipLaunchKernelGGL(k_heads_bwd<bf16_t>, grid, dim3(GATE_NTHR), 0, st, tokens, H, H * E, m.R, m.U,
                       (int)m.nbg, (const bf16_t*)x, (const bf16_t*)xb, A, b, dg, dbeta, (bf16_t*)dx,
                       (bf16_t*)dxb, part);
  else
    hipLaunchKernelGGL(k_heads_bwd<float>, grid, dim3(GATE_NTHR), 0, st, tokens, H, H * E, m.R, m.U,
                       (int)m.nbg, (const float*)x, (const float*)xb, A, b, dg, dbeta, (float*)dx,
                       (float*)dxb, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_heads_sum, dim3(H * E), dim3(GATE_NTHR), 0, st, (int)m.nbg, H * E, part, dA, db);
  return hipGetLastError();
}


template <typename T>
static hipError_t gate_fwd_t(long long rows, int V, const void* o, const void* z, const float* w,
                             float eps, void* y, hipStream_t st) {
  const int nb = gate_grid(rows, V, 4096);
#define GATE_F(V_)                                                                                  \
  case V_:                                                                                          \
    hipLaunchKernelGGL((k_gate_fwd<T, V_>), dim3(nb), dim3(GATE_NTHR), 0, st, rows, (const T*)o,    \
                       (const T*)z, w, eps, (T*)y);                                                 \
    break;
  switch (V) {
    GATE_F(16) GATE_F(32) GATE_F(64) GATE_F(128) GATE_F(256)
    default: return hipErrorInvalidValue;
  }
#undef GATE_F
  return hipGetLastError();
}

template <typename T>
static hipError_t gate_bwd_t(long long rows, int V, const void* o, const void* z, const float* w,
                             float eps, const void* dy, void* d_o, void* dz, float* dw_part,
                             hipStream_t st) {
  const int nb = gate_blocks(rows, V);
#define GATE_B(V_)                                                                                  \
  case V_:                                                                                          \
    hipLaunchKernelGGL((k_gate_bwd<T, V_>), dim3(nb), dim3(GATE_NTHR), 0, st, rows, (const T*)o,    \
                       (const T*)z, w, eps, (const T*)dy, (T*)d_o, (T*)dz, dw_part);                \
    break;
  switch (V) {
    GATE_B(16) GATE_B(32) GATE_B(64) GATE_B(128) GATE_B(256)
    default: return hipErrorInvalidValue;
  }
#undef GATE_B
  return hipGetLastError();
}

hipError_t launch_gate_fwd(bool bf16, long long rows, int V, const void* o, const void* z,
                           const float* w, float eps, void* y, hipStream_t st) {
  return bf16 ? gate_fwd_t<bf16_t>(rows, V, o, z, w, eps, y, st)
              : gate_fwd_t<float>(rows, V, o, z, w, eps, y, st);
}

hipError_t launch_gate_bwd(bool bf16, long long rows, int V, const void* o, const void* z,
                           const float* w, float eps, const void* dy, void* d_o, void* dz,
                           float* dw_part, hipStream_t st) {
  return bf16 ? gate_bwd_t<bf16_t>(rows, V, o, z, w, eps, dy, d_o, dz, dw_part, st)
              : gate_bwd_t<float>(rows, V, o, z, w, eps, dy, d_o, dz, dw_part, st);
}

hipError_t launch_gate_dw(long long rows, int V, const float* dw_part, float* dw, hipStream_t st) {
  hipLaunchKernelGGL(k_gate_dw, dim3(V), dim3(GATE_NTHR), 0, st, gate_blocks(rows, V), V, dw_part, dw);
  return hipGetLastError();
}

}  // namespace tla
