// Recurrent single-token decode step (Eq. forget3 / Eq. gdn3, read of Eq. la3).
//
// One pass over the fp32 state: each workgroup owns VC value columns of one
// (sequence, head) for all E*K rows.  Every thread loads its rows (128-byte
// row segments per 8 lanes), decays them by the slice gate, accumulates the
// retrieval r = kappa^T Sbar and the read-out rho^T Sbar with the joint key
// kappa = k2 (x) k and joint query rho = q2 (x) q, and keeps the rows in
// registers.  After a fixed-order workgroup reduction it forms
//   w = beta (v - r)   (GDN)   or   beta v   (sGLA)
//   o = rho^T Sbar + (q2 . k2)(q . k) w        (= rho^T S_t)
// and writes S_t = Sbar + kappa w^T back: one read and one write of the state,
// both nontemporal (the state streams through once per step).
#include "tla_common.hpp"
#include "tla_internal.hpp"

namespace tla {

template <typename T, int KD, int E, int VC, int NTHR>
__global__ __launch_bounds__(NTHR) void k_step(Shape s, FwdIn in, float* state, void* out) {
  constexpr int TPR = VC / 4;            // threads per row (float4 each)
  constexpr int NRG = NTHR / TPR;        // row groups
  constexpr int ROWS = E * KD;
  constexpr int RPT = ROWS / NRG;        // rows per thread
  static_assert(RPT * NRG == ROWS, "rows must split evenly");
  constexpr int NSUM = 2 * VC;           // (quantity, column) sums
  constexpr int TPS = NTHR / NSUM;       // threads per sum
  static_assert(TPS >= 1 && TPS <= 64 && (64 % TPS) == 0, "reduction shape");

  __shared__ float sk[KD], sq[KD], sk2[E], sq2[E], sa[E], sv[VC], sw[VC];
  __shared__ float sdot[2];
  __shared__ f32x4 red[2][NRG][TPR];
  __shared__ float tot[NSUM];

  const int tid = threadIdx.x;
  const int V = s.V;
  const int nct = V / VC;
  int nh, ct;
  xcd_map(blockIdx.x, s.NH, nct, nh, ct);
  const int c0 = ct * VC;
  const T* qg = (const T*)in.q + (size_t)nh * KD;
  const T* kg = (const T*)in.k + (size_t)nh * KD;
  const T* vg = (const T*)in.v + (size_t)nh * V + c0;
  const T* q2g = (const T*)in.q2 + (size_t)nh * E;
  const T* k2g = (const T*)in.k2 + (size_t)nh * E;
  const float* gg = in.g + (size_t)nh * E;

  for (int i = tid; i < KD; i += NTHR) {
    sk[i] = ld_f(kg + i);
    sq[i] = ld_f(qg + i);
  }
  for (int i = tid; i < E; i += NTHR) {
    sk2[i] = ld_f(k2g + i);
    sq2[i] = ld_f(q2g + i);
    sa[i] = __expf(gg[i]);
  }
  for (int i = tid; i < VC; i += NTHR) sv[i] = ld_f(vg + i);
  if (tid < 64) {  // (q . k) and (q2 . k2) for the current token's own write
    float a = 0.f, c = 0.f;
    for (int i = tid; i < KD; i += 64) a += ld_f(qg + i) * ld_f(kg + i);
    for (int i = tid; i < E; i += 64) c += ld_f(q2g + i) * ld_f(k2g + i);
    a = wave_sum(a);
    c = wave_sum(c);
    if (tid == 0) {
      sdot[0] = a;
      sdot[1] = c;
    }
  }
  __syncthreads();

  const int p = tid % TPR, rg = tid / TPR;
  float* base = state + (size_t)nh * ROWS * V + c0 + 4 * p;
  f32x4 st[RPT];
  f32x4 racc = zero4(), oacc = zero4();
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int row = rg + NRG * i;
    st[i] = __builtin_nontemporal_load((const f32x4*)(base + (size_t)row * V));
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int row = rg + NRG * i;
    const int e = row / KD, kd = row % KD;
    st[i] *= sa[e];
    racc += (sk2[e] * sk[kd]) * st[i];
    oacc += (sq2[e] * sq[kd]) * st[i];
  }
  red[0][rg][p] = racc;
  red[1][rg][p] = oacc;
  __syncthreads();
  {  // fixed-order reduction over the row groups: TPS threads per (quantity, column)
    const int sidx = tid / TPS, part = tid % TPS;
    const int qn = sidx / VC, col = sidx % VC;
    float acc = 0.f;
    for (int r = part; r < NRG; r += TPS) acc += red[qn][r][col / 4][col % 4];
#pragma unroll
    for (int o = TPS / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (part == 0) tot[sidx] = acc;
  }
  __syncthreads();
  if (tid < VC) {
    const int col = tid;
    const float bt = in.beta ? in.beta[nh] : 1.f;
    const float w = (s.variant == 1) ? bt * (sv[col] - tot[col]) : bt * sv[col];
    const float o = tot[VC + col] + sdot[0] * sdot[1] * w;
    sw[col] = w;
    const size_t off = (size_t)nh * V + c0 + col;
    if (s.out_bf16)
      ((bf16_t*)out)[off] = Elem<bf16_t>::from_f(o);
    else
      ((float*)out)[off] = o;
  }
  __syncthreads();
  const f32x4 w4 = *(const f32x4*)&sw[4 * p];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int row = rg + NRG * i;
    const int e = row / KD, kd = row % KD;
    const f32x4 x = st[i] + (sk2[e] * sk[kd]) * w4;
    __builtin_nontemporal_store(x, (f32x4*)(base + (size_t)row * V));
  }
}

template <typename T, int KD, int E, int VC>
static hipError_t step_inst(const Shape& s, const FwdIn& in, float* state, void* o, hipStream_t st) {
  constexpr int ROWS = E * KD;
  constexpr int TPR = VC / 4;
  constexpr int WANT = ROWS * TPR;  // threads for one row each
  constexpr int NTHR = WANT < 1024 ? WANT : 1024;
  hipLaunchKernelGGL((k_step<T, KD, E, VC, NTHR>), dim3(s.NH * (s.V / VC)), dim3(NTHR), 0, st, s,
                     in, state, o);
  return hipGetLastError();
}

template <typename T, int KD, int E>
static hipError_t step_vc(const Shape& s, const FwdIn& in, float* state, void* o, hipStream_t st) {
  if (s.V % 32 == 0) return step_inst<T, KD, E, 32>(s, in, state, o, st);
  return step_inst<T, KD, E, 16>(s, in, state, o, st);
}

#define TLA_STEP_CASE(KD_, E_)                                             \
  if (s.K == KD_ && s.E == E_) {                                           \
    if (s.in_bf16) return step_vc<bf16_t, KD_, E_>(s, in, state, o, st);   \
    return step_vc<float, KD_, E_>(s, in, state, o, st);                   \
  }

hipError_t launch_step(const Shape& s, const FwdIn& in, float* state, void* o, hipStream_t st) {
  TLA_STEP_CASE(16, 4)
  TLA_STEP_CASE(32, 4)
  TLA_STEP_CASE(32, 32)
  TLA_STEP_CASE(64, 8)
  TLA_STEP_CASE(64, 16)
  TLA_STEP_CASE(128, 1)
  TLA_STEP_CASE(128, 4)
  TLA_STEP_CASE(128, 8)
  TLA_STEP_CASE(128, 16)
  return hipErrorInvalidValue;
}

}  // namespace tla
