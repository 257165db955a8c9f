// Forward of chunkwise triadic linear attention on gfx950.
//
//   k_prep  one workgroup per (head, chunk), chunk-parallel:
//           in-chunk cumulative log-gates G (Appendix A: gamma^r_e is the
//           product of the slice's gates over positions 1..r), the row
//           coefficient vectors a_e = k'_e o gamma_e, b_e = q'_e o gamma_e,
//           c_e = k'_e o gamma^C_e / gamma_e, gamma^C_e; A_qk = Q K^T and
//           A_kk = K K^T on MFMA; the decayed second-key Grams R (Eq.
//           joint-gram) and R' formed element by element from exponentials of
//           non-positive log-gate differences (Appendix A, numerical
//           stability); M = A_qk o R'; and the UT transform
//           Tu = (I + tril(diag(beta)(A_kk o R), -1))^{-1} diag(beta)
//           (Eq. joint-solve) by a blocked fp32 unit-lower inverse.
//   k_fwd   one workgroup per (head, 16-column value tile), sequential over
//           chunks (Eq. joint-chunk).  The E x K x 16 fp32 state tile lives
//           in MFMA accumulators for the whole sequence; each wave owns
//           E / waves slices.  Per chunk:
//             P^K_e = K S_e,  P^Q_e = Q S_e                     (MFMA)
//             W = sum_e diag(a_e) P^K_e                         (LDS reduce)
//             U = Tu (V - W)   [GDN]   or   diag(beta) V  [sGLA]
//             O = sum_e diag(b_e) P^Q_e + M U
//             S_e <- gamma^C_e S_e + K^T diag(c_e) U            (MFMA)
//           Tu is applied to the residual (no per-slice W = T K precompute).
//           Value columns never interact (Eq. slices), which is what makes
//           the 16-column tiling exact.
#include "tla_common.hpp"
#include "tla_internal.hpp"

namespace tla {

template <typename T>
__device__ __forceinline__ void copy8(T* dst, const T* src) {
  if constexpr (sizeof(T) == 2) {
    *(uint4*)dst = *(const uint4*)src;
  } else {
    ((float4*)dst)[0] = ((const float4*)src)[0];
    ((float4*)dst)[1] = ((const float4*)src)[1];
  }
}
template <typename T>
__device__ __forceinline__ void zero8(T* dst) {
  if constexpr (sizeof(T) == 2) {
    *(uint4*)dst = make_uint4(0, 0, 0, 0);
  } else {
    ((float4*)dst)[0] = make_float4(0, 0, 0, 0);
    ((float4*)dst)[1] = make_float4(0, 0, 0, 0);
  }
}

// Contraction over a D-deep axis given fragment accessors for A and B.
// fa(kb) / fb(kb) return the 16-deep fragment of block kb.
template <int D, typename FA, typename FB>
__device__ __forceinline__ void mma_k(f32x4& acc, FA fa, FB fb) {
  constexpr int NB = D / 16;
#pragma unroll
  for (int kb = 0; kb + 1 < NB; kb += 2) mma32(acc, fa(kb), fa(kb + 1), fb(kb), fb(kb + 1));
  if constexpr (NB & 1) mma16(acc, fa(NB - 1), fb(NB - 1));
}

// ------------------------------------------------------------------- prep
// LDS plan: Q and K rows (bf16 instances) share their space with the inverse
// of (I + L) and its scratch, which are formed after the Grams.
//
// Every operand tile leaves as whole 128-byte lines (eight consecutive
// elements per lane, consecutive lanes along a row) with the nontemporal
// hint: the recurrent kernel that runs next reads these tiles once, and
// partly written lines left dirty in L2 were written back while it ran
// (measured 40-50 us slower at B4 H8 T4096).  M leaves from a row-major
// copy of it (LINES), Tu from the inverse; K^T and Q^T are read out of the
// staged rows column-wise.  Instances whose plan would then exceed two
// workgroups per CU keep the per-tile stores.
template <typename T, int KD, int C, int E>
struct PrepSmem {
  static constexpr int KP = KD + 8;  // 16-byte rows, conflict-free 16-byte fragment reads
  static constexpr int CP = C + 4;
  static constexpr int NT = C / 16;
  static constexpr bool STAGE = sizeof(T) == 2;  // fp32 rows are read from global memory
  static constexpr size_t plan_bytes(bool lines) {
    const size_t qk = 2 * (STAGE ? C : 1) * KP * sizeof(T) + (lines ? C * CP * 4 : 0);
    const size_t inv = C * CP * 4 + (NT > 1 ? NT - 1 : 1) * 16 * 17 * 4;
    return (qk > inv ? qk : inv) + C * CP * 4 + 2 * C * E * 4 + C * E * 8 + C * 4 + 64;
  }
  static constexpr bool LINES = STAGE && plan_bytes(true) <= 80 * 1024;
  union U {
    struct {
      T sQ[STAGE ? C : 1][KP];
      T sK[STAGE ? C : 1][KP];
      float Mb[LINES ? C : 1][CP];  // M, for the line-wise stores
    } qk;
    struct { float X[C][CP]; float Y[NT > 1 ? NT - 1 : 1][16][17]; } inv;
  };
  alignas(16) U u;
  alignas(16) float L[C][CP];  // diag(beta)(A_kk o R), strictly lower
  alignas(16) float q2[C][E];
  alignas(16) float k2[C][E];
  alignas(16) double G[C][E];  // in-chunk cumulative log-gates
  alignas(16) float beta[C];
};

// Eight waves per chunk for E <= 8: two workgroups fit a CU (the
// shared-memory plan), so each phase's work is split over twice the waves
// that four would give; larger E keeps four (their registers would not fit
// 128 per lane).
template <int E> constexpr int prep_waves() { return E <= 8 ? 8 : 4; }

// Eight consecutive values of a bf16 (hi, lo) operand tile: the high parts
// at dst, the low parts one matrix (C x C elements) further, one 16-byte
// nontemporal store each.
template <int C>
__device__ __forceinline__ void store8_split(bf16_t* dst, f32x4 x0, f32x4 x1) {
  bf16x4 h0, l0, h1, l1;
  split_frag(x0, h0, l0);
  split_frag(x1, h1, l1);
  gstore_b128(dst, __builtin_bit_cast(u32x4, __builtin_shufflevector(h0, h1, 0, 1, 2, 3, 4, 5, 6, 7)));
  gstore_b128(dst + C * C, __builtin_bit_cast(u32x4, __builtin_shufflevector(l0, l1, 0, 1, 2, 3, 4, 5, 6, 7)));
}

template <typename T, int KD, int C, int E>
__global__ __launch_bounds__(prep_waves<E>() * 64) void k_prep(Shape s, FwdIn in, PrepBufs p) {
  constexpr int PREP_NW = prep_waves<E>();
  constexpr int PREP_NTHR = PREP_NW * 64;
  constexpr int NT = C / 16;
  constexpr int E4 = (E + 3) & ~3;
  typedef PrepSmem<T, KD, C, E> Sm;
  constexpr bool STAGE = Sm::STAGE;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Sm& sm = *reinterpret_cast<Sm*>(smem_raw);

  const int ch = blockIdx.x;
  const int head = ch / s.Nc, ci = ch % s.Nc;
  const int b = head / s.H, h = head % s.H;
  const int t0 = ci * C;
  const int tid = threadIdx.x;
  const size_t tok0 = seq_begin(s, b);
  s.T = seq_len(s, b);  // this sequence's length from here on
  if (t0 >= s.T) return;  // past the end of a shorter packed sequence
  const int w = wave_id(), l = lane_id(), g = l >> 4, n = l & 15;
  const size_t krs = (size_t)s.H * KD;
  const T* Qg = (const T*)in.q + (tok0 * s.H + h) * KD;
  const T* Kg = (const T*)in.k + (tok0 * s.H + h) * KD;
  const size_t eoff = (tok0 * s.H + h) * E, erow = (size_t)s.H * E;

  // ---- per-position vectors; Q and K rows (rows past T read clamped, then
  // zeroed).  Every global load of the phase is issued before the first of
  // their results is stored (one memory latency instead of one per array).
  constexpr int NQE = (C * E + PREP_NTHR - 1) / PREP_NTHR;  // q2, k2 entries per thread
  constexpr int IT = STAGE ? (C * KD / 8 + PREP_NTHR - 1) / PREP_NTHR : 1;
  constexpr int NGE = (E + PREP_NW - 1) / PREP_NW;  // slices per wave (g)
  float q2v[NQE], k2v[NQE], bv = 0.f;
  Raw8<T> qv[IT], kv[IT];
  double gv[NGE];
#pragma unroll
  for (int i = 0; i < NQE; ++i) {
    const int idx = min(tid + PREP_NTHR * i, C * E - 1), r = idx / E, e = idx % E;
    const size_t off = eoff + (size_t)min(t0 + r, s.T - 1) * erow + e;
    q2v[i] = ld_f((const T*)in.q2 + off);
    k2v[i] = ld_f((const T*)in.k2 + off);
  }
  if (tid < C) {
    const int t = min(t0 + tid, s.T - 1);
    bv = in.beta ? in.beta[(tok0 + t) * s.H + h] : 1.f;
  }
  if constexpr (STAGE) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = min(tid + PREP_NTHR * it, C * KD / 8 - 1);
      const int r = idx / (KD / 8), c8 = idx % (KD / 8);
      const size_t off = (size_t)min(t0 + r, s.T - 1) * krs + 8 * c8;
      qv[it] = load8(Qg + off);
      kv[it] = load8(Kg + off);
    }
  }
#pragma unroll
  for (int i = 0; i < NGE; ++i) {
    const int e = min(w + PREP_NW * i, E - 1);
    gv[i] = (double)in.g[eoff + (size_t)min(t0 + l, s.T - 1) * erow + e];
  }
  // ---- the stores
#pragma unroll
  for (int i = 0; i < NQE; ++i) {
    const int idx = tid + PREP_NTHR * i, r = idx / E, e = idx % E;
    if (idx >= C * E) continue;
    const bool ok = t0 + r < s.T;
    sm.q2[r][e] = ok ? q2v[i] : 0.f;
    sm.k2[r][e] = ok ? k2v[i] : 0.f;
  }
  if (tid < C) sm.beta[tid] = (t0 + tid < s.T) ? bv : 0.f;
  if constexpr (STAGE) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + PREP_NTHR * it;
      if (idx >= C * KD / 8) continue;
      const int r = idx / (KD / 8), c8 = idx % (KD / 8);
      const bool ok = t0 + r < s.T;
      *(Raw8<T>*)&sm.u.qk.sQ[r][8 * c8] = ok ? qv[it] : zero_raw8<T>();
      *(Raw8<T>*)&sm.u.qk.sK[r][8 * c8] = ok ? kv[it] : zero_raw8<T>();
    }
  }
  // G: inclusive cumulative sum over the chunk in fp64 (one wave per slice,
  // lane r holds row r); after a very negative gate the running sum is large
  // and fp32 would lose the small gates that follow it
#pragma unroll
  for (int i = 0; i < NGE; ++i) {
    const int e = w + PREP_NW * i;
    if (e >= E) continue;  // wave-uniform
    double x = (l < C && t0 + l < s.T) ? gv[i] : 0.0;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double y = __shfl_up(x, off, 64);
      if (l >= off) x += y;
    }
    if (l < C) sm.G[l][e] = x;
  }
  __syncthreads();

  // ---- coefficient vectors a = k2 gamma, b = q2 gamma, c = k2 gamma^C / gamma; gamma^C
  float* coef = p.coef + (size_t)ch * 3 * E * C;
  for (int idx = tid; idx < E * C / 4; idx += PREP_NTHR) {  // four consecutive positions per thread
    const int e = idx / (C / 4), r0 = 4 * (idx % (C / 4));
    const double GC = sm.G[C - 1][e];
    f32x4 a, bq, c;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const double G = sm.G[r0 + j][e];
      const float gam = exp_nonpos((float)G);
      a[j] = sm.k2[r0 + j][e] * gam;
      bq[j] = sm.q2[r0 + j][e] * gam;
      c[j] = sm.k2[r0 + j][e] * exp_nonpos((float)(GC - G));
    }
    gstore_b128(coef + (0 * E + e) * C + r0, __builtin_bit_cast(u32x4, a));
    gstore_b128(coef + (1 * E + e) * C + r0, __builtin_bit_cast(u32x4, bq));
    gstore_b128(coef + (2 * E + e) * C + r0, __builtin_bit_cast(u32x4, c));
  }
  if (tid < E4) p.gC[(size_t)ch * E4 + tid] = (tid < E) ? exp_nonpos((float)sm.G[C - 1][tid]) : 0.f;

  // ---- 16 x 16 tiles: A_qk, A_kk on MFMA, then per lane (rows 16 rt + 4 g + j,
  // column 16 st + n) the decayed Grams R', R, M = A_qk o R' (r >= c) and
  // L = diag(beta)(A_kk o R) (r > c); tiles above the diagonal are zero
  auto qrow8 = [&](int r, int col) -> Raw8<T> {
    if (col >= KD) return zero_raw8<T>();
    if constexpr (STAGE) {
      return *(const Raw8<T>*)&sm.u.qk.sQ[r][col];
    } else {
      const Raw8<T> x = load8(Qg + (size_t)min(t0 + r, s.T - 1) * krs + col);
      return (t0 + r < s.T) ? x : zero_raw8<T>();
    }
  };
  auto krow8 = [&](int r, int col) -> Raw8<T> {
    if (col >= KD) return zero_raw8<T>();
    if constexpr (STAGE) {
      return *(const Raw8<T>*)&sm.u.qk.sK[r][col];
    } else {
      const Raw8<T> x = load8(Kg + (size_t)min(t0 + r, s.T - 1) * krs + col);
      return (t0 + r < s.T) ? x : zero_raw8<T>();
    }
  };
  typedef OpTiles<T, KD, C> OT;
  T* ops = (T*)p.ops + (size_t)ch * OT::STRIDE;
  // M tile (rt, st) of the lane layout into the row-major copy, split into
  // (hi, lo) for bf16 operands
  auto put_m = [&](int rt, int st, f32x4 mv) {
    f32x4 parts[2];
    if constexpr (OT::NS == 2) {
      parts[0] = bf16x4_to_f(cvt_frag<bf16_t>(mv));
      parts[1] = mv - parts[0];
    } else {
      parts[0] = mv;
    }
#pragma unroll
    for (int pt = 0; pt < OT::NS; ++pt) {
      store_tile16(ops + OT::M + pt * OT::MAT + (size_t)(16 * rt) * C + 16 * st, parts[pt], g, n, C);
    }
  };
  for (int tile = w; tile < NT * NT; tile += PREP_NW) {
    constexpr int NL = NT * (NT + 1) / 2;  // lower tiles first, then the upper ones
    int rt = 0, st = 0;
    if (tile < NL) {
      while ((rt + 1) * (rt + 2) / 2 <= tile) ++rt;
      st = tile - rt * (rt + 1) / 2;
    } else {
      int u = tile - NL;
      while (u >= NT - 1 - rt) {
        u -= NT - 1 - rt;
        ++rt;
      }
      st = rt + 1 + u;
    }
    const int c = 16 * st + n;
    if (st > rt) {
#pragma unroll
      for (int j = 0; j < 4; ++j) sm.L[16 * rt + 4 * g + j][c] = 0.f;
      if constexpr (Sm::LINES) {
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.u.qk.Mb[16 * rt + 4 * g + j][c] = 0.f;
      } else {
        put_m(rt, st, zero4());
      }
      continue;
    }
    f32x4 aq = zero4(), ak = zero4();
#pragma unroll
    for (int kp = 0; kp < (KD + 31) / 32; ++kp) {
      const int col = 32 * kp + 8 * g;
      const Raw8<T> kb = krow8(c, col);
      mma8(aq, qrow8(16 * rt + n, col), kb);
      mma8(ak, krow8(16 * rt + n, col), kb);
    }
    // (every pair of the tile is formed and masked afterwards: no per-lane
    // branch around the shared-memory reads, which are whole-row vector reads)
    double Gc[E];
    float k2c[E];
    lds_row<E>(Gc, &sm.G[c][0]);
    lds_row<E>(k2c, &sm.k2[c][0]);
    f32x4 mv;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = 16 * rt + 4 * g + j;
      double Gr[E];
      float q2r[E], k2r[E];
      lds_row<E>(Gr, &sm.G[r][0]);
      lds_row<E>(q2r, &sm.q2[r][0]);
      lds_row<E>(k2r, &sm.k2[r][0]);
      float rq = 0.f, rk = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float d = exp_nonpos((float)(Gr[e] - Gc[e])) * k2c[e];
        rq += q2r[e] * d;
        rk += k2r[e] * d;
      }
      mv[j] = (c <= r) ? aq[j] * rq : 0.f;
      sm.L[r][c] = (c < r) ? sm.beta[r] * ak[j] * rk : 0.f;
    }
    if constexpr (Sm::LINES) {
#pragma unroll
      for (int j = 0; j < 4; ++j) sm.u.qk.Mb[16 * rt + 4 * g + j][c] = mv[j];
    } else {
      put_m(rt, st, mv);
    }
  }
  // ---- M, K^T (and for the backward Q^T) as whole lines
  if constexpr (Sm::LINES) {
    __syncthreads();  // M complete
    for (int idx = tid; idx < C * C / 8; idx += PREP_NTHR) {
      const int r = idx / (C / 8), c8 = 8 * (idx % (C / 8));
      const float* src = &sm.u.qk.Mb[r][c8];
      store8_split<C>(ops + OT::M + (size_t)r * C + c8, *(const f32x4*)src, *(const f32x4*)(src + 4));
    }
    // row R of K^T holds key key_of_row(R); column c position row_of_key(c)
    // (the key orders of the recurrent kernels' state tiles)
    const int nmat = p.bwd_tiles ? 2 : 1;
    for (int idx = tid; idx < nmat * KD * C / 8; idx += PREP_NTHR) {
      const int mtx = idx / (KD * C / 8), rem = idx % (KD * C / 8);
      const int R = rem / (C / 8), c8 = 8 * (rem % (C / 8));
      const int key = key_of_row<KD>(R);
      uint32_t wd[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p0 = row_of_key<C>(c8 + 2 * i), p1 = row_of_key<C>(c8 + 2 * i + 1);
        const uint16_t v0 = mtx ? sm.u.qk.sQ[p0][key] : sm.u.qk.sK[p0][key];
        const uint16_t v1 = mtx ? sm.u.qk.sQ[p1][key] : sm.u.qk.sK[p1][key];
        wd[i] = (uint32_t)v0 | ((uint32_t)v1 << 16);
      }
      gstore_b128(ops + (mtx ? OT::Qt : OT::Kt) + (size_t)R * C + c8,
                  u32x4{wd[0], wd[1], wd[2], wd[3]});
    }
  } else {  // K^T (and for the backward Q^T) of the chunk (4 x 4 blocks; rows
            // past T are zero)
    constexpr int NB = (C / 4) * (KD / 4);
    const int nmat = p.bwd_tiles ? 2 : 1;
    for (int idx = tid; idx < nmat * NB; idx += PREP_NTHR) {
      const int mtx = idx / NB, bi = idx % NB;
      const int rb = bi / (KD / 4), kb = bi % (KD / 4);
      float x[4][4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * rb + i;
        if constexpr (STAGE) {
          const T* src = mtx ? &sm.u.qk.sQ[r][4 * kb] : &sm.u.qk.sK[r][4 * kb];
#pragma unroll
          for (int j = 0; j < 4; ++j) x[i][j] = Elem<T>::to_f(src[j]);
        } else {
          const T* src = (mtx ? Qg : Kg) + (size_t)min(t0 + r, s.T - 1) * krs + 4 * kb;
          const bool ok = t0 + r < s.T;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float v = Elem<T>::to_f(src[j]);
            x[i][j] = ok ? v : 0.f;
          }
        }
      }
      // (rows in the key order of the recurrent kernels' state tiles: key k
      // at row row_of_key(k); positions in the same order within 32-blocks,
      // position r at column key_of_row(r), so that the eight positions of a
      // lane group's 32-deep operand (4 g + j and 16 + 4 g + j) are adjacent;
      // both keep each group of four together)
      T* dst = ops + (mtx ? OT::Qt : OT::Kt);
      const int row4 = row_of_key<KD>(4 * kb), col4 = key_of_row<C>(4 * rb);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        put4<T>(dst + (size_t)(row4 + j) * C + col4, f32x4{x[0][j], x[1][j], x[2][j], x[3][j]});
    }
  }
  __syncthreads();

  // ---- Tu = (I + L)^{-1} diag(beta) (GDN), blocked unit-lower inverse in fp32
  if (s.variant == 1) {
    unit_lower_inverse<C, PREP_NTHR>([&](int r, int c) { return sm.L[r][c]; }, &sm.u.inv.X[0][0],
                               Sm::CP, &sm.u.inv.Y[0][0][0]);
    if (p.ninv) {  // kept in fp32 for the backward of the solve
      float* dst = p.ninv + (size_t)ch * C * C;
      for (int idx = tid; idx < C * C / 4; idx += PREP_NTHR) {
        const int r = idx / (C / 4), c4 = idx % (C / 4);
        gstore_b128(dst + r * C + 4 * c4, __builtin_bit_cast(u32x4, *(const f32x4*)&sm.u.inv.X[r][4 * c4]));
      }
    }
    if constexpr (Sm::LINES) {  // Tu = X diag(beta), row-major
      for (int idx = tid; idx < C * C / 8; idx += PREP_NTHR) {
        const int r = idx / (C / 8), c8 = 8 * (idx % (C / 8));
        const float* src = &sm.u.inv.X[r][c8];
        store8_split<C>(ops + OT::Tu + (size_t)r * C + c8, *(const f32x4*)src * *(const f32x4*)&sm.beta[c8],
                     *(const f32x4*)(src + 4) * *(const f32x4*)&sm.beta[c8 + 4]);
      }
    } else
    // Tu row-major, from 4 x 4 blocks of the inverse
    for (int idx = tid; idx < (C / 4) * (C / 4); idx += PREP_NTHR) {
      const int rb = idx / (C / 4), cb = idx % (C / 4);
      const f32x4 bc = *(const f32x4*)&sm.beta[4 * cb];
      f32x4 x[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) x[i] = *(const f32x4*)&sm.u.inv.X[4 * rb + i][4 * cb] * bc;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (OT::NS == 2) {
          const f32x4 hr = bf16x4_to_f(cvt_frag<bf16_t>(x[i]));
          put4<T>(ops + OT::Tu + (size_t)(4 * rb + i) * C + 4 * cb, hr);
          put4<T>(ops + OT::Tu + OT::MAT + (size_t)(4 * rb + i) * C + 4 * cb, x[i] - hr);
        } else {
          put4<T>(ops + OT::Tu + (size_t)(4 * rb + i) * C + 4 * cb, x[i]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------- forward
// PK (the forward with state and output waves at E = 16): two key slices
// share one 16-column accumulator tile, 8 value columns each; the W and O
// partials are then stored once per value column (32 lanes).
template <typename T, int KD, int C, int E, int NW, bool PK = false>
struct FwdSmem {
  static constexpr int NT = C / 16;
  static constexpr int E4 = (E + 3) & ~3;
  static constexpr int EC = 16 / (int)sizeof(T);
  // bf16 operands carry Tu and M as hi + lo pairs (SPLIT).  The largest
  // instances read the queries straight from global memory so that the plan
  // fits the 160 KiB of LDS.
  static constexpr bool SPLIT = sizeof(T) == 2;
  static constexpr bool STAGE_Q = sizeof(T) == 2 && (E < 16 || PK);
  static constexpr int PL = PK ? 32 : 64;  // lanes of a partial-sum tile
  SwzTile<T, C, KD> K;
  SwzTile<T, STAGE_Q ? C : 1, STAGE_Q ? KD : EC> Q;
  SwzTile<T, KD, C> Kt;
  SwzTile<T, C, C> Tu, M;
  SwzTile<T, SPLIT ? C : 1, SPLIT ? C : EC> TuL, ML;
  // V tile rows, permuted within each 16-row block: position 16 b + 4 j + i
  // holds row 16 b + 4 i + j, so that the four rows 4 i + j (i = 0..3) a
  // lane group reads together are adjacent (no bank conflicts)
  alignas(16) T Vr[C][16];
  alignas(16) float coef01[2][E][C];  // a_e, b_e
  alignas(16) float coef2[E][C];      // c_e
  alignas(16) float gC[E4];
  alignas(16) float beta[C];
  alignas(16) f32x4 W[NW][NT][PL];
  alignas(16) f32x4 O[NW][NT][PL];
  alignas(16) f32x4 Us[NT][64];  // U row tiles in the accumulator layout
};

// Direct copies of one chunk's operands into shared memory, in four groups
// issued at different points of a chunk step (each right after the barrier
// that frees its destination):
//   KQ  the K (and Q) rows and the coefficients a_e, b_e   (for the next chunk)
//   Tu  Tu (hi, lo)                                         (for the next chunk)
//   M   M (hi, lo)                                          (for the next chunk)
//   Kt  K^T and the coefficients c_e                        (for this chunk)
// Wave w copies the 1 KiB blocks w, w + NW, ... of a tile, where w is the
// wave's index within its group of NW waves (the forward with separate state
// and output waves has two groups of four, each issuing its own copies).  K
// and Q rows past
// T are read from row T - 1 (and zeroed after arrival in the last chunk);
// M, Tu and K^T come from the prep kernel's operand tiles, whose rows and
// columns past T are already zero.
template <typename T, int KD, int C, int E, int NW, bool PK = false>
struct FwdDma : GroupDma<NW> {
  typedef GroupDma<NW> G;
  typedef FwdSmem<T, KD, C, E, NW, PK> Sm;
  typedef OpTiles<T, KD, C> OT;
  using G::tile;
  using G::wid;
  template <typename Tile>
  static constexpr int tile_count() { return G::template tile_count<Tile>(); }
  template <int NBYTES>
  static constexpr int co_count() { return G::template co_count<NBYTES>(); }
  template <int NBYTES>
  static __device__ __forceinline__ void copy(void* dst, const void* src) {
    G::template copy<NBYTES>(dst, src);
  }
  template <typename Tile>
  static __device__ __forceinline__ void op_tile(Tile& t, const T* src) {
    G::template op_tile<C>(t, src);
  }
  static constexpr int NCO01 = 2 * E * C * 4, NCO2 = E * C * 4;  // bytes
  static constexpr int N_KQ = tile_count<decltype(Sm::K)>() +
                              (Sm::STAGE_Q ? tile_count<decltype(Sm::Q)>() : 0) + co_count<NCO01>();
  static constexpr int N_TU = tile_count<decltype(Sm::Tu)>() * (Sm::SPLIT ? 2 : 1);
  static constexpr int N_M = tile_count<decltype(Sm::M)>() * (Sm::SPLIT ? 2 : 1);
  static constexpr int N_KT = tile_count<decltype(Sm::Kt)>() + co_count<NCO2>();
  static constexpr int N_KC = tile_count<decltype(Sm::K)>() + co_count<NCO01>();
  static constexpr int N_Q = tile_count<decltype(Sm::Q)>();
  static __device__ __forceinline__ void kq(Sm& sm, const Shape& s, const PrepBufs& p, const T* Kg,
                                            const T* Qg, size_t ch, int t0) {
    const size_t krs = (size_t)s.H * KD;
    const int last = s.T - 1 - t0;  // rows past it are read from row T - 1
    auto off = [=](int r, int c) {
      return (uint32_t)(sizeof(T) * ((size_t)min(r, last) * krs + Sm::EC * c));
    };
    tile(sm.K, Kg + (size_t)t0 * krs, off);
    if constexpr (Sm::STAGE_Q) tile(sm.Q, Qg + (size_t)t0 * krs, off);
    copy<NCO01>(&sm.coef01[0][0][0], p.coef + ch * 3 * E * C);
  }
  // K rows with a_e, b_e (N_KC copies) and Q rows (N_Q copies) separately
  static __device__ __forceinline__ void kc(Sm& sm, const Shape& s, const PrepBufs& p, const T* Kg,
                                            size_t ch, int t0) {
    const size_t krs = (size_t)s.H * KD;
    const int last = s.T - 1 - t0;
    tile(sm.K, Kg + (size_t)t0 * krs, [=](int r, int c) {
      return (uint32_t)(sizeof(T) * ((size_t)min(r, last) * krs + Sm::EC * c));
    });
    copy<NCO01>(&sm.coef01[0][0][0], p.coef + ch * 3 * E * C);
  }
  static __device__ __forceinline__ void q(Sm& sm, const Shape& s, const T* Qg, int t0) {
    const size_t krs = (size_t)s.H * KD;
    const int last = s.T - 1 - t0;
    tile(sm.Q, Qg + (size_t)t0 * krs, [=](int r, int c) {
      return (uint32_t)(sizeof(T) * ((size_t)min(r, last) * krs + Sm::EC * c));
    });
  }
  static __device__ __forceinline__ void tu(Sm& sm, const PrepBufs& p, size_t ch) {
    const T* ops = (const T*)p.ops + ch * OT::STRIDE;
    op_tile(sm.Tu, ops + OT::Tu);
    if constexpr (Sm::SPLIT) op_tile(sm.TuL, ops + OT::Tu + OT::MAT);
  }
  static __device__ __forceinline__ void m(Sm& sm, const PrepBufs& p, size_t ch) {
    const T* ops = (const T*)p.ops + ch * OT::STRIDE;
    op_tile(sm.M, ops + OT::M);
    if constexpr (Sm::SPLIT) op_tile(sm.ML, ops + OT::M + OT::MAT);
  }
  static __device__ __forceinline__ void kt(Sm& sm, const PrepBufs& p, size_t ch) {
    const T* ops = (const T*)p.ops + ch * OT::STRIDE;
    op_tile(sm.Kt, ops + OT::Kt);
    copy<NCO2>(&sm.coef2[0][0], p.coef + ch * 3 * E * C + 2 * E * C);
  }

  // The copies below are exactly one instruction per wave, so that every
  // wave's vmcnt waits can count them.
  // gamma^C of the chunk (every wave copies the same E4 values)
  static __device__ __forceinline__ void gc(Sm& sm, const PrepBufs& p, size_t ch) {
    if (lane_id() < Sm::E4) lds_dma<4>(p.gC + ch * Sm::E4, 4 * lane_id(), lds_addr(&sm.gC[0]));
  }
  // The V tile (rows t0 .. t0 + C - 1, the workgroup's 16 columns) in the
  // permuted row order of Sm::Vr; wave w copies 16-byte pieces
  // [w VL, (w + 1) VL) of the tile.  Rows past T read row T - 1 (zeroed after
  // arrival in the last chunk).  Vg points at the columns' start in row t0.
  // PK: the workgroup's 8 columns fill both halves of each row.
  static constexpr int PPR = 16 * (int)sizeof(T) / 16;  // 16-byte pieces per row
  static constexpr int VL = C * PPR / NW;                // lanes per wave
  static_assert(C * PPR % NW == 0 && VL <= 64, "V tile split over the waves");
  static __device__ __forceinline__ void v(Sm& sm, const T* Vg, size_t vrs, int last) {
    const int w = wid(), l = lane_id();
    const int q = w * VL + l, pos = q / PPR, part = q % PPR;
    const int r = (pos & ~15) + 4 * (pos & 3) + ((pos >> 2) & 3);  // row held at position pos
    const uint32_t off = (uint32_t)(sizeof(T) * (size_t)min(r, last) * vrs) + (PK ? 0 : 16 * part);
    if (l < VL) lds_dma<16>(Vg, off, lds_addr(&sm.Vr[0][0]) + 16 * w * VL);
  }
  // beta of the chunk's rows (sGLA with beta), rows past T read row T - 1;
  // bg points at the beta of row t0 (row stride H)
  static constexpr int BL = C / NW;
  static __device__ __forceinline__ void beta(Sm& sm, const float* bg, int H, int last) {
    const int w = wid(), l = lane_id();
    const uint32_t off = (uint32_t)(4 * (size_t)min(w * BL + l, last) * H);
    if (l < BL) lds_dma<4>(bg, off, lds_addr(&sm.beta[0]) + 4 * w * BL);
  }
};

template <typename T, int KD, int C, int E, int NW>
__global__ __launch_bounds__(NW * 64) void k_fwd(Shape s, FwdIn in, PrepBufs p, void* out,
                                                 float* s_final, SavedBufs sv, int train) {
  constexpr int SPW = (E + NW - 1) / NW;
  constexpr bool RAGGED = E % NW != 0;  // some waves own fewer slices
  constexpr int NT = C / 16;
  constexpr int KT = KD / 16;
  constexpr int NTHR = NW * 64;
  typedef typename Elem<T>::frag F;
  typedef FwdSmem<T, KD, C, E, NW> Sm;
  typedef FwdDma<T, KD, C, E, NW> Dma;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Sm& sm = *reinterpret_cast<Sm*>(smem_raw);

  const int w = wave_id(), l = lane_id(), g = l >> 4, n = l & 15;
  const int V = s.V;
  int head, vt;
  xcd_map(blockIdx.x, s.NH, V / 16, head, vt);
  const int b = head / s.H, h = head % s.H;
  const int v0 = vt * 16;
  const size_t tok0 = seq_begin(s, b);
  s.T = seq_len(s, b);                 // this sequence's length from here on
  const int nc = (s.T + C - 1) / C;    // its chunks (s.Nc: the per-head stride)

  // state tiles S[i][kt] = S_e[16 kt + 4 g + j][v0 + n], e = w * SPW + i
  f32x4 S[SPW][KT];
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const int e = w * SPW + i;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      f32x4 x = zero4();
      if (in.s0 && e < E) {
        const float* src = in.s0 + (((size_t)head * E + e) * KD + key_col<KD>(kt, g)) * V + v0 + n;
#pragma unroll
        for (int j = 0; j < 4; ++j) x[j] = src[(size_t)j * V];
      }
      S[i][kt] = x;
    }
  }

  const T* Kg = (const T*)in.k + (tok0 * s.H + h) * KD;
  const T* Qg = (const T*)in.q + (tok0 * s.H + h) * KD;
  const T* Vg = (const T*)in.v + (tok0 * s.H + h) * (size_t)V + v0;
  const size_t krs = (size_t)s.H * KD;  // row stride between positions
  const size_t ch0 = (size_t)head * s.Nc;

  const bf16x4 idf = identity_frag();  // for the transposing checkpoint stores
  const size_t vrs = (size_t)s.H * V;
  const bool sbeta = s.variant == 0 && in.beta != nullptr;  // beta copied per chunk
  const float* bg = in.beta ? in.beta + tok0 * s.H + h : nullptr;
  if (s.variant == 0 && !in.beta)
    for (int r = threadIdx.x; r < C; r += NTHR) sm.beta[r] = 1.f;
  if (nc > 0) {
    Dma::kq(sm, s, p, Kg, Qg, ch0, 0);
    Dma::v(sm, Vg, vrs, s.T - 1);
    if (sbeta) Dma::beta(sm, bg, s.H, s.T - 1);
    Dma::tu(sm, p, ch0);
    Dma::m(sm, p, ch0);
  }
  // Vector memory operations this wave issues after the gamma^C copy and
  // before the wait that precedes the state update (all of them exactly
  // counted): checkpoint tile stores, the next chunk's K, Q rows and a_e,
  // b_e, the X and U stores, the next chunk's Tu, V tile and beta.  The wait
  // then covers the K^T, c_e and gamma^C copies without waiting for the
  // stores.  (A compiler-issued load among them would only make it stricter.)
  const int owned = RAGGED ? max(0, min(SPW, E - w * SPW)) : SPW;
  const int n_st = (train ? owned * KT : 0) + ((train && w < NT) ? (s.variant == 1 ? 8 : 4) : 0);
  const int n_more = n_st + Dma::N_KQ + Dma::N_TU + 1 + (sbeta ? 1 : 0);

  for (int ci = 0; ci < nc; ++ci) {
    const int t0 = ci * C;
    const size_t ch = ch0 + ci;
    const bool more = ci + 1 < nc;
    __syncthreads();  // the previous chunk is done with K^T, c_e and gamma^C

    Dma::kt(sm, p, ch);
    Dma::gc(sm, p, ch);
    // the K, Q rows, a_e, b_e, Tu, M, V tile and beta of this chunk have
    // landed (only the K^T, c_e and gamma^C copies just issued may still be
    // in flight)
    wait_vmcnt<Dma::N_KT + 1>();
    if (t0 + C > s.T) {  // every wave's copies must have landed before the zeroing
      __syncthreads();
      zero_rows_from(sm.K, s.T - t0, NTHR);
      if constexpr (Sm::STAGE_Q) zero_rows_from(sm.Q, s.T - t0, NTHR);
      for (int pos = threadIdx.x; pos < C; pos += NTHR) {
        const int r = (pos & ~15) + 4 * (pos & 3) + ((pos >> 2) & 3);
        if (t0 + r >= s.T)
          for (int c = 0; c < 16; ++c) sm.Vr[pos][c] = T(0);
      }
    }
    __syncthreads();

    // ---- operand copies of the chunk-start state
    F Sop[SPW][KT];
#pragma unroll
    for (int i = 0; i < SPW; ++i)
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) Sop[i][kt] = cvt_frag<T>(S[i][kt]);

    if (train) {  // chunk-start state for the backward: [ch][E][V/16][K][16]
#pragma unroll
      for (int i = 0; i < SPW; ++i) {
        const int e = w * SPW + i;
        if (RAGGED && e >= E) continue;
        T* dst = (T*)sv.Sck + ((ch * E + e) * (size_t)(V / 16) + vt) * KD * 16;
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
          if constexpr (sizeof(T) == 2)
            store_tile16_frag(dst + 256 * kt, Sop[i][kt], idf, g, n);
          else
            store_tile16(dst + 256 * kt, S[i][kt], g, n);
        }
      }
    }

    // ---- P^K_e = K S_e, then P^Q_e = Q S_e for the owned slices, each folded
    // straight into this wave's partial of W = sum_e diag(a_e) P^K_e and of
    // sum_e diag(b_e) P^Q_e (the two passes keep one set of accumulators live)
    {
      // The 32-deep A operand of K (pass 0) or Q (pass 1) rows for row tile
      // rt and the key blocks kb, kb + 1 (kb even): keys key_col(kb, g) ..
      // + 7, one 16-byte piece of the row in the key order of the state tiles
      auto afrag8 = [&](int pass, int rt, int kb) -> Frag8<T> {
        const int r = 16 * rt + n, c = key_col<KD>(kb, g);
        Frag8<T> f;
        if constexpr (sizeof(T) == 2) {
          if (pass == 0) {
            f.v = *(const bf16x8*)sm.K.at(r, c);
          } else if constexpr (Sm::STAGE_Q) {
            f.v = *(const bf16x8*)sm.Q.at(r, c);
          } else {
            const bool qok = t0 + r < s.T;
            const uint4 x = qok ? *(const uint4*)(Qg + (size_t)(t0 + r) * krs + c) : make_uint4(0, 0, 0, 0);
            f.v = __builtin_bit_cast(bf16x8, x);
          }
        } else {
          if (pass == 0) {
            f.lo = ld_frag(sm.K.at(r, c));
            f.hi = ld_frag(sm.K.at(r, c + 4));
          } else if constexpr (Sm::STAGE_Q) {
            f.lo = ld_frag(sm.Q.at(r, c));
            f.hi = ld_frag(sm.Q.at(r, c + 4));
          } else {
            const bool qok = t0 + r < s.T;
            f.lo = qok ? ld_frag(Qg + (size_t)(t0 + r) * krs + c) : zero4();
            f.hi = qok ? ld_frag(Qg + (size_t)(t0 + r) * krs + c + 4) : zero4();
          }
        }
        return f;
      };
      // A fragment of K (pass 0) or Q (pass 1) rows for row tile rt, block kb
      // (16-deep, for a single key block)
      auto afrag = [&](int pass, int rt, int kb) -> F {
        const int r = 16 * rt + n;
        if (pass == 0) return ld_frag(sm.K.at(r, key_col<KD>(kb, g)));
        if constexpr (Sm::STAGE_Q) {
          return ld_frag(sm.Q.at(r, key_col<KD>(kb, g)));
        } else {
          const bool qok = t0 + r < s.T;
          return qok ? ld_frag(Qg + (size_t)(t0 + r) * krs + key_col<KD>(kb, g)) : cvt_frag<T>(zero4());
        }
      };
      // fold the accumulators of a pass into this wave's partial
      auto fold = [&](int pass, f32x4(&P)[SPW][NT]) {
#pragma unroll
        for (int rt = 0; rt < NT; ++rt) {
          f32x4 acc = zero4();
#pragma unroll
          for (int i = 0; i < SPW; ++i) {
            const int e = w * SPW + i;
            if (RAGGED && e >= E) continue;
            acc += *(const f32x4*)&sm.coef01[pass][e][16 * rt + 4 * g] * P[i][rt];
          }
          if (pass == 0)
            sm.W[w][rt][l] = acc;
          else
            sm.O[w][rt][l] = acc;
        }
      };
      constexpr bool PIPE = KT > 1 && NW <= 4;
      if constexpr (PIPE) {
        // steps j = 0 .. 2 NS - 1 over (pass, k-block pair); the fragments of
        // step j + 1 are loaded before the MFMAs of step j, so the shared
        // memory latency hides behind them (with one wave per SIMD nothing
        // else would; two waves per SIMD hide it for each other and have no
        // registers to spare).  NT x SPW independent accumulators advance per
        // step.
        constexpr int NS = KT / 2;
        auto load_step = [&](int j, Frag8<T>(&x)[NT]) {
          const int ps = j / NS, kb = 2 * (j % NS);
#pragma unroll
          for (int rt = 0; rt < NT; ++rt) x[rt] = afrag8(ps, rt, kb);
        };
        f32x4 P[SPW][NT];
#pragma unroll
        for (int rt = 0; rt < NT; ++rt)
#pragma unroll
          for (int i = 0; i < SPW; ++i) P[i][rt] = zero4();
        Frag8<T> a[NT];
        load_step(0, a);
#pragma unroll
        for (int j = 0; j < 2 * NS; ++j) {
          Frag8<T> bn[NT];
          if (j + 1 < 2 * NS) load_step(j + 1, bn);
          const int kb = 2 * (j % NS);
#pragma unroll
          for (int i = 0; i < SPW; ++i) {
            if (RAGGED && w * SPW + i >= E) continue;
#pragma unroll
            for (int rt = 0; rt < NT; ++rt) mma32(P[i][rt], a[rt], Sop[i][kb], Sop[i][kb + 1]);
          }
          if (j % NS == NS - 1) {
            fold(j / NS, P);
#pragma unroll
            for (int rt = 0; rt < NT; ++rt)
#pragma unroll
              for (int i = 0; i < SPW; ++i) P[i][rt] = zero4();
          }
          if (j + 1 < 2 * NS) {
#pragma unroll
            for (int rt = 0; rt < NT; ++rt) a[rt] = bn[rt];
          }
        }
      } else {
        // k-block outer: the fragments of all row tiles are loaded together
        // and NT x SPW independent accumulators advance per step
#pragma unroll
        for (int pass = 0; pass < 2; ++pass) {
          f32x4 P[SPW][NT];
#pragma unroll
          for (int rt = 0; rt < NT; ++rt)
#pragma unroll
            for (int i = 0; i < SPW; ++i) P[i][rt] = zero4();
#pragma unroll
          for (int kb = 0; kb < KT; kb += (KT > 1 ? 2 : 1)) {
            if constexpr (KT > 1) {
              Frag8<T> a[NT];
#pragma unroll
              for (int rt = 0; rt < NT; ++rt) a[rt] = afrag8(pass, rt, kb);
#pragma unroll
              for (int i = 0; i < SPW; ++i) {
                if (RAGGED && w * SPW + i >= E) continue;
#pragma unroll
                for (int rt = 0; rt < NT; ++rt) mma32(P[i][rt], a[rt], Sop[i][kb], Sop[i][kb + 1]);
              }
            } else {
              F a[NT];
#pragma unroll
              for (int rt = 0; rt < NT; ++rt) a[rt] = afrag(pass, rt, 0);
#pragma unroll
              for (int i = 0; i < SPW; ++i) {
                if (RAGGED && w * SPW + i >= E) continue;
#pragma unroll
                for (int rt = 0; rt < NT; ++rt) mma16(P[i][rt], a[rt], Sop[i][0]);
              }
            }
          }
          fold(pass, P);
        }
      }
    }
    __syncthreads();
    // K, Q rows and a_e, b_e are free: the next chunk's are copied while this
    // chunk computes
    if (more) Dma::kq(sm, s, p, Kg, Qg, ch + 1, t0 + C);

    // ---- U = Tu (V - W) (GDN) or diag(beta) V (sGLA): wave w < NT forms row
    // tile w and the tiles are exchanged through LDS.  Every block kb of the
    // row is formed, also those right of the diagonal (Tu is zero there, so
    // they add exact zeros): no branch separates the shared-memory reads, so
    // they are all in flight before the first one is used.
    // rows 16 kb + 4 g + j of the lane's value column, j = 0..3
    auto vrows = [&](int kb) {
      f32x4 x;
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = Elem<T>::to_f(sm.Vr[16 * kb + 4 * j + g][n]);
      return x;
    };
    if (w < NT) {
      const int rt = w;
      f32x4 u;
      if (s.variant == 1) {
        const int r = 16 * rt + n;
        f32x4 xr[NT], wq[NW][NT];
        F th[NT], tl[NT];
        T vr[NT][4];  // raw V elements (converted after the reads are issued)
#pragma unroll
        for (int kb = 0; kb < NT; ++kb) {
#pragma unroll
          for (int j = 0; j < 4; ++j) vr[kb][j] = sm.Vr[16 * kb + 4 * j + g][n];
#pragma unroll
          for (int ww = 0; ww < NW; ++ww) wq[ww][kb] = sm.W[ww][kb][l];
          th[kb] = ld_frag(sm.Tu.at(r, 16 * kb + 4 * g));
          if constexpr (Sm::SPLIT) tl[kb] = ld_frag(sm.TuL.at(r, 16 * kb + 4 * g));
        }
        // (keeps the reads above together: the scheduler would otherwise
        // interleave each with its use and wait for every one in turn)
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kb = 0; kb < NT; ++kb) {
#pragma unroll
          for (int j = 0; j < 4; ++j) xr[kb][j] = Elem<T>::to_f(vr[kb][j]);
#pragma unroll
          for (int ww = 0; ww < NW; ++ww) xr[kb] -= wq[ww][kb];
        }
        F Xh[NT], Xl[NT];
        f32x4 xd = xr[0];  // the diagonal block, saved for the backward
#pragma unroll
        for (int kb = 0; kb < NT; ++kb) {
          split_frag(xr[kb], Xh[kb], Xl[kb]);
          if (kb > 0 && kb == rt) xd = xr[kb];
        }
        if (train) {
          float* dst = sv.X + ch * C * (size_t)V + (size_t)(16 * rt + 4 * g) * V + v0 + n;
#pragma unroll
          for (int j = 0; j < 4; ++j) gstore_b32(dst + (size_t)j * V, __float_as_uint(xd[j]));
        }
        u = zero4();
#pragma unroll
        for (int kb = 0; kb < NT; kb += (NT > 1 ? 2 : 1)) {
          if constexpr (NT > 1) {
            mma32(u, th[kb], th[kb + 1], Xh[kb], Xh[kb + 1]);
            if constexpr (Sm::SPLIT) {
              mma32(u, th[kb], th[kb + 1], Xl[kb], Xl[kb + 1]);
              mma32(u, tl[kb], tl[kb + 1], Xh[kb], Xh[kb + 1]);
            }
          } else {
            mma16(u, th[0], Xh[0]);
            if constexpr (Sm::SPLIT) {
              mma16(u, th[0], Xl[0]);
              mma16(u, tl[0], Xh[0]);
            }
          }
        }
      } else {
        u = vrows(rt) * *(const f32x4*)&sm.beta[16 * rt + 4 * g];
      }
      sm.Us[rt][l] = u;
      if (train) {
        float* dst = sv.U + ch * C * (size_t)V + (size_t)(16 * rt + 4 * g) * V + v0 + n;
#pragma unroll
        for (int j = 0; j < 4; ++j) gstore_b32(dst + (size_t)j * V, __float_as_uint(u[j]));
      }
    }
    __syncthreads();
    if (more) {  // Tu, the V tile and beta are free
      Dma::tu(sm, p, ch + 1);
      Dma::v(sm, Vg + (size_t)(t0 + C) * vrs, vrs, s.T - 1 - (t0 + C));
      if (sbeta) Dma::beta(sm, bg + (size_t)(t0 + C) * s.H, s.H, s.T - 1 - (t0 + C));
    }
    f32x4 U[NT];
    F Uh[NT], Ul[NT];
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) {
      U[rt] = sm.Us[rt][l];
      split_frag(U[rt], Uh[rt], Ul[rt]);
    }

    // ---- O for row tile w: sum of the partials plus M U
    f32x4 oacc = zero4();
    if (w < NT) {
      const int rt = w;
      const int r = 16 * rt + n;
      F mf[NT], ml[NT];  // all fragment reads first
#pragma unroll
      for (int kb = 0; kb < NT; ++kb) {
        mf[kb] = ld_frag(sm.M.at(r, 16 * kb + 4 * g));
        if constexpr (Sm::SPLIT) ml[kb] = ld_frag(sm.ML.at(r, 16 * kb + 4 * g));
      }
      f32x4 op[NW];
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) op[ww] = sm.O[ww][rt][l];
      __builtin_amdgcn_sched_barrier(0);  // the reads above stay together
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) oacc += op[ww];
      mma_k<C>(oacc, [&](int kb) { return mf[kb]; }, [&](int kb) { return Uh[kb]; });
      if constexpr (Sm::SPLIT) {
        mma_k<C>(oacc, [&](int kb) { return mf[kb]; }, [&](int kb) { return Ul[kb]; });
        mma_k<C>(oacc, [&](int kb) { return ml[kb]; }, [&](int kb) { return Uh[kb]; });
      }
    }
    // K^T, c_e and gamma^C of this chunk have landed (n_more / n_st count
    // what was issued after them); every wave is done with M after the barrier
    wait_vmcnt_rt(more ? n_more : n_st);
    __syncthreads();
    if (more) Dma::m(sm, p, ch + 1);
    if (w < NT) {
      const int rt = w;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = t0 + 16 * rt + 4 * g + j;
        if (t < s.T) {
          const size_t off = ((tok0 + t) * s.H + h) * (size_t)V + v0 + n;
          if (s.out_bf16)
            ((bf16_t*)out)[off] = Elem<bf16_t>::from_f(oacc[j]);
          else
            ((float*)out)[off] = oacc[j];
        }
      }
    }

    // ---- state update S_e <- gamma^C_e S_e + K^T diag(c_e) U
    F Uc[SPW][NT], Ucl[SPW][NT];
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int e = w * SPW + i;
      if (RAGGED && e >= E) continue;
      const float gc = sm.gC[e];
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) S[i][kt] *= gc;
#pragma unroll
      for (int kb = 0; kb < NT; ++kb)
        split_frag(U[kb] * *(const f32x4*)&sm.coef2[e][16 * kb + 4 * g], Uc[i][kb], Ucl[i][kb]);
    }
    // k-block outer: KT x SPW independent accumulators per step
#pragma unroll
    for (int kb = 0; kb < NT; kb += (NT > 1 ? 2 : 1)) {
      if constexpr (NT > 1) {
        // K^T rows: positions 4 g + j and 16 + 4 g + j of the block pair are
        // adjacent in the operand tile (one 16-byte read per lane)
        Frag8<T> a[KT];
        const int c = key_of_row<C>(16 * kb + 4 * g);
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
          if constexpr (sizeof(T) == 2) {
            a[kt].v = *(const bf16x8*)sm.Kt.at(16 * kt + n, c);
          } else {
            a[kt].lo = ld_frag(sm.Kt.at(16 * kt + n, c));
            a[kt].hi = ld_frag(sm.Kt.at(16 * kt + n, c + 4));
          }
        }
#pragma unroll
        for (int i = 0; i < SPW; ++i) {
          if (RAGGED && w * SPW + i >= E) continue;
#pragma unroll
          for (int kt = 0; kt < KT; ++kt) mma32(S[i][kt], a[kt], Uc[i][kb], Uc[i][kb + 1]);
          if constexpr (Sm::SPLIT) {
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) mma32(S[i][kt], a[kt], Ucl[i][kb], Ucl[i][kb + 1]);
          }
        }
      } else {
        F a[KT];
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) a[kt] = ld_frag(sm.Kt.at(16 * kt + n, 4 * g));
#pragma unroll
        for (int i = 0; i < SPW; ++i) {
          if (RAGGED && w * SPW + i >= E) continue;
#pragma unroll
          for (int kt = 0; kt < KT; ++kt) {
            mma16(S[i][kt], a[kt], Uc[i][0]);
            if constexpr (Sm::SPLIT) mma16(S[i][kt], a[kt], Ucl[i][0]);
          }
        }
      }
    }
  }

  if (s_final) {
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int e = w * SPW + i;
      if (RAGGED && e >= E) continue;
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        float* dst = s_final + (((size_t)head * E + e) * KD + key_col<KD>(kt, g)) * V + v0 + n;
#pragma unroll
        for (int j = 0; j < 4; ++j) dst[(size_t)j * V] = S[i][kt][j];
      }
    }
  }
}

// ------------------------------------------- forward with state and output waves
// The same chunk step on eight waves in two roles.  Waves 0..3 (state waves)
// own E/4 slices of the state each, in fp32 registers, and run only what the
// next chunk waits for: their partial of W = sum_e diag(a_e) K S_e, U
// (Tu (V - W) for GDN, diag(beta) V for sGLA) and the update
// S_e <- gamma^C_e S_e + K^T diag(c_e) U of the chunkwise form (Appendix A,
// Eq. joint-chunk).
// After each update they leave the bf16 operand copy of the new state in
// shared memory.  Waves 4..7 (output waves; wave 4 + i shares a SIMD with
// state wave i) take it from there and form the chunk's output rows,
// sum_e diag(b_e) Q S_e + M U, and its checkpoint, in the shadow of the
// state waves' work.  Three barriers divide a chunk step:
//   B0 .. B1  state: K S_e, W partials          output: Q S_e partials
//   B1 .. B2  state: U, one row tile per wave   output: rows of V - W
//   B2 .. B0  state: the update                 output: O rows (partials + M U)
// The output waves issue every global store (checkpoint, U, V - W, O).
// The state waves issue and await every copy into shared memory (also Q and
// M, which only the output waves read), and the output waves never wait for
// memory: a wave's vmcnt wait for a copy also waits for the stores it issued
// before the copy, which under the write traffic of all workgroups take
// thousands of cycles to be acknowledged.
template <typename T, int KD, int C, int E, bool PK = false>
struct DualSmem {
  FwdSmem<T, KD, C, E, 4, PK> f;
  // bf16 operand copy of the chunk-start state: [slice (PK: slice pair)][key
  // tile][lane], each lane's entry as the state wave's lane holds it
  alignas(16) typename Elem<T>::frag sop[PK ? E / 2 : E][KD / 16][64];
};

// PK (inference at E = 16, K = 128): the workgroup owns 8 value columns and
// each accumulator tile holds two key slices side by side (columns 0..7:
// slice 2 u, columns 8..15: slice 2 u + 1 of "unit" u), so that the per-unit
// work and shared memory match the E = 8 instance and the long-context
// shape (few heads) launches twice the workgroups.  The row coefficients
// then differ between the two column halves of a tile, and the W and O
// partials are summed over the halves (a DPP rotation by 8 lanes).  The
// U tile is formed with both halves holding the same 8 columns (V is copied
// into both).  No checkpoints: training forwards keep the 16-column kernel.
template <typename T, int KD, int C, int E, bool PK = false>
__global__ __launch_bounds__(512) void k_fwd_dual(Shape s, FwdIn in, PrepBufs p, void* out,
                                                  float* s_final, SavedBufs sv, int train) {
  constexpr int NG = 4;  // waves per role
  constexpr int UE = PK ? E / 2 : E;  // slices or slice pairs
  constexpr int SPW = UE / NG;
  constexpr int NT = C / 16;
  constexpr int KT = KD / 16;
  constexpr int NTHR = 2 * NG * 64;
  constexpr int VW = PK ? 8 : 16;     // value columns of a workgroup
  static_assert(UE % NG == 0 && sizeof(T) == 2, "bf16 operands, whole slices per wave");
  typedef typename Elem<T>::frag F;
  typedef FwdSmem<T, KD, C, E, NG, PK> Sm;
  typedef FwdDma<T, KD, C, E, NG, PK> Dma;
  static_assert(Sm::STAGE_Q && Sm::SPLIT, "queries staged, Tu and M as hi + lo pairs");
  extern __shared__ __align__(16) unsigned char smem_raw[];
  DualSmem<T, KD, C, E, PK>& smd = *reinterpret_cast<DualSmem<T, KD, C, E, PK>*>(smem_raw);
  Sm& sm = smd.f;
  if constexpr (PK) train = 0;

  const int wv = wave_id(), w = wv & (NG - 1), l = lane_id(), g = l >> 4, n = l & 15;
  const int V = s.V;
  int head, vt;
  xcd_map(blockIdx.x, s.NH, V / VW, head, vt);
  const int b = head / s.H, h = head % s.H;
  const int v0 = vt * VW;
  // the key slice and value column of this lane in unit i of its wave
  const int vc = PK ? (n & 7) : n;
  auto slc = [&](int i) { return PK ? 2 * (w * SPW + i) + (n >> 3) : w * SPW + i; };
  const int pl = PK ? 8 * g + (n & 7) : l;  // this lane's entry of a partial-sum tile
  const size_t tok0 = seq_begin(s, b);
  s.T = seq_len(s, b);                 // this sequence's length from here on
  const int nc = (s.T + C - 1) / C;    // its chunks (s.Nc: the per-head stride)

  const T* Kg = (const T*)in.k + (tok0 * s.H + h) * KD;
  const T* Qg = (const T*)in.q + (tok0 * s.H + h) * KD;
  const T* Vg = (const T*)in.v + (tok0 * s.H + h) * (size_t)V + v0;
  const size_t ch0 = (size_t)head * s.Nc;
  const size_t vrs = (size_t)s.H * V;
  const bool sbeta = s.variant == 0 && in.beta != nullptr;  // beta copied per chunk
  const float* bg = in.beta ? in.beta + tok0 * s.H + h : nullptr;
  if (s.variant == 0 && !in.beta)
    for (int r = threadIdx.x; r < C; r += NTHR) sm.beta[r] = 1.f;

  // Rows past T of the last, partial chunk: every copy of both roles has
  // landed, then the K, Q and V rows are zeroed (run by all waves).
  auto zero_tail = [&](int t0) {
    wait_vmcnt<0>();
    __syncthreads();
    zero_rows_from(sm.K, s.T - t0, NTHR);
    zero_rows_from(sm.Q, s.T - t0, NTHR);
    for (int pos = threadIdx.x; pos < C; pos += NTHR) {
      const int r = (pos & ~15) + 4 * (pos & 3) + ((pos >> 2) & 3);
      if (t0 + r >= s.T)
        for (int c = 0; c < 16; ++c) sm.Vr[pos][c] = T(0);
    }
    __syncthreads();
  };

  // X S_e for the wave's slices (X: the chunk's K or Q rows), folded with the
  // coefficient vectors cf[e] (a_e or b_e) into the wave's partial dst[rt][l].
  // The fragments of the next k-block pair are read before the MFMAs of the
  // current one.
  auto state_pass = [&](const decltype(sm.K)& X, const F(&So)[SPW][KT], const float(*cf)[C],
                        f32x4(*dst)[Sm::PL]) {
    f32x4 P[SPW][NT];
#pragma unroll
    for (int i = 0; i < SPW; ++i)
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) P[i][rt] = zero4();
    if constexpr (KT > 1) {
      constexpr int NS = KT / 2;
      auto load = [&](int j, Frag8<T>(&a)[NT]) {
#pragma unroll
        for (int rt = 0; rt < NT; ++rt) a[rt].v = *(const bf16x8*)X.at(16 * rt + n, key_col<KD>(2 * j, g));
      };
      Frag8<T> a[NT];
      load(0, a);
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        Frag8<T> bn[NT];
        if (j + 1 < NS) load(j + 1, bn);
#pragma unroll
        for (int i = 0; i < SPW; ++i)
#pragma unroll
          for (int rt = 0; rt < NT; ++rt) mma32(P[i][rt], a[rt], So[i][2 * j], So[i][2 * j + 1]);
        if (j + 1 < NS) {
#pragma unroll
          for (int rt = 0; rt < NT; ++rt) a[rt] = bn[rt];
        }
      }
    } else {
      F a[NT];
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) a[rt] = ld_frag(X.at(16 * rt + n, 4 * g));
#pragma unroll
      for (int i = 0; i < SPW; ++i)
#pragma unroll
        for (int rt = 0; rt < NT; ++rt) mma16(P[i][rt], a[rt], So[i][0]);
    }
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) {
      f32x4 acc = zero4();
#pragma unroll
      for (int i = 0; i < SPW; ++i) acc += *(const f32x4*)&cf[slc(i)][16 * rt + 4 * g] * P[i][rt];
      if constexpr (PK) {  // the two slices of each unit: columns n and n + 8
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] += dpp_f<0x128>(acc[j]);  // row_ror:8
        if (n < 8) dst[rt][pl] = acc;
      } else {
        dst[rt][l] = acc;
      }
    }
  };

  // The checkpoint (the chunk-start state for the backward,
  // [ch][E][V/16][K][16]) of the slices of wave w goes out in NPC pieces of
  // one 16-byte store per lane.  A piece is a pair of key tiles (1 KiB): lane
  // o = 16 grp + 4 q + r writes row 4 grp + r of tile q / 2 of the pair,
  // columns 8 (q & 1) .. + 7, which two transposing reads of the
  // register-order copy give it (as source, lane 16 grp + 4 j + q reads
  // state-wave lane 16 grp + 8 (q & 1) + j, and + 4, of tile q / 2).  With an
  // odd number of key tiles a piece is one tile, transposed on the matrix
  // cores.
  constexpr bool PAIRS = KT % 2 == 0;
  constexpr int NPC = PAIRS ? SPW * KT / 2 : SPW * KT;
  constexpr int KH = PAIRS ? KT / 2 : 1;  // key tile pairs
  // data of piece pc, read from the copy of the chunk-start state
  auto piece_read = [&](int pc) -> u32x4 {
    const int sq = l & 3, e = w * SPW + pc / KH, kt = 2 * (pc % KH) + (sq >> 1);
    const F* src = &smd.sop[e][kt][16 * (l >> 4) + 8 * (sq & 1) + ((l & 15) >> 2)];
    const bf16x4 a = lds_read_tr16(src), b = lds_read_tr16(src + 4);
    return __builtin_bit_cast(u32x4, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  auto piece_store = [&](size_t ch, int pc, u32x4 d) {
    const int oq = (l & 15) >> 2, i = pc / KH, kt = 2 * (pc % KH) + (oq >> 1);
    T* dst = (T*)sv.Sck + ((ch * E + w * SPW + i) * (size_t)(V / 16) + vt) * KD * 16;
    gstore_b128(dst + 256 * kt + 16 * (4 * (l >> 4) + (l & 3)) + 8 * (oq & 1), d);
  };

  if (wv < NG) {
    // ================================================= state waves
    // S[i][kt] = S_e[key_col(kt, g) + j][v0 + n], e = w SPW + i
    f32x4 S[SPW][KT];
    F Sop[SPW][KT];
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int e = slc(i);
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        f32x4 x = zero4();
        if (in.s0) {
          const float* src = in.s0 + (((size_t)head * E + e) * KD + key_col<KD>(kt, g)) * V + v0 + vc;
#pragma unroll
          for (int j = 0; j < 4; ++j) x[j] = src[(size_t)j * V];
        }
        S[i][kt] = x;
        Sop[i][kt] = cvt_frag<T>(x);
        smd.sop[w * SPW + i][kt][l] = Sop[i][kt];
      }
    }
    if (nc > 0) {
      Dma::kc(sm, s, p, Kg, ch0, 0);
      Dma::q(sm, s, Qg, 0);
      Dma::tu(sm, p, ch0);
      Dma::v(sm, Vg, vrs, s.T - 1);
      if (sbeta) Dma::beta(sm, bg, s.H, s.T - 1);
      wait_vmcnt_rt(Dma::N_TU + 1 + (sbeta ? 1 : 0));  // K, Q, a_e, b_e have landed
    }

    for (int ci = 0; ci < nc; ++ci) {
      const int t0 = ci * C;
      const size_t ch = ch0 + ci;
      const bool more = ci + 1 < nc;
      __syncthreads();  // B0
      if (t0 + C > s.T) zero_tail(t0);
      Dma::kt(sm, p, ch);
      Dma::gc(sm, p, ch);
      Dma::m(sm, p, ch);

      // ---- W partial: sum over the wave's slices of diag(a_e) K S_e (GDN;
      // sGLA has no W)
      if (s.variant == 1) state_pass(sm.K, Sop, sm.coef01[0], sm.W[w]);
      wait_vmcnt<Dma::N_KT + 1 + Dma::N_M>();  // this chunk's Tu, V and beta have landed
      __syncthreads();  // B1
      if (more) {  // K, Q, a_e and b_e are free
        Dma::kc(sm, s, p, Kg, ch + 1, t0 + C);
        Dma::q(sm, s, Qg, t0 + C);
      }

      // ---- U for row tile w: Tu (V - W) (GDN) or diag(beta) V (sGLA).  Every
      // block kb of the row is formed (Tu is zero right of the diagonal), so no
      // branch separates the shared-memory reads.
      if (w < NT) {
        const int rt = w;
        f32x4 u;
        if (s.variant == 1) {
          const int r = 16 * rt + n;
          f32x4 xr[NT], wq[NG][NT];
          F th[NT], tl[NT];
          T vr[NT][4];
#pragma unroll
          for (int kb = 0; kb < NT; ++kb) {
#pragma unroll
            for (int j = 0; j < 4; ++j) vr[kb][j] = sm.Vr[16 * kb + 4 * j + g][n];
#pragma unroll
            for (int ww = 0; ww < NG; ++ww) wq[ww][kb] = sm.W[ww][kb][pl];
            th[kb] = ld_frag(sm.Tu.at(r, 16 * kb + 4 * g));
            tl[kb] = ld_frag(sm.TuL.at(r, 16 * kb + 4 * g));
          }
          __builtin_amdgcn_sched_barrier(0);  // the reads above stay together
#pragma unroll
          for (int kb = 0; kb < NT; ++kb) {
#pragma unroll
            for (int j = 0; j < 4; ++j) xr[kb][j] = Elem<T>::to_f(vr[kb][j]);
#pragma unroll
            for (int ww = 0; ww < NG; ++ww) xr[kb] -= wq[ww][kb];
          }
          F Xh[NT], Xl[NT];
#pragma unroll
          for (int kb = 0; kb < NT; ++kb) split_frag(xr[kb], Xh[kb], Xl[kb]);
          u = zero4();
#pragma unroll
          for (int kb = 0; kb < NT; kb += (NT > 1 ? 2 : 1)) {
            if constexpr (NT > 1) {
              mma32(u, th[kb], th[kb + 1], Xh[kb], Xh[kb + 1]);
              mma32(u, th[kb], th[kb + 1], Xl[kb], Xl[kb + 1]);
              mma32(u, tl[kb], tl[kb + 1], Xh[kb], Xh[kb + 1]);
            } else {
              mma16(u, th[0], Xh[0]);
              mma16(u, th[0], Xl[0]);
              mma16(u, tl[0], Xh[0]);
            }
          }
        } else {
          f32x4 x;
#pragma unroll
          for (int j = 0; j < 4; ++j) x[j] = Elem<T>::to_f(sm.Vr[16 * rt + 4 * j + g][n]);
          u = x * *(const f32x4*)&sm.beta[16 * rt + 4 * g];
        }
        sm.Us[rt][l] = u;
      }
      // K^T, c_e, gamma^C and M have landed (immediate counts: a wait with a
      // count known only at run time costs a chain of scalar branches)
      if (more)
        wait_vmcnt<Dma::N_KC + Dma::N_Q>();
      else
        wait_vmcnt<0>();
      __syncthreads();  // B2
      if (more) {  // Tu, the V tile and beta are free
        Dma::tu(sm, p, ch + 1);
        Dma::v(sm, Vg + (size_t)(t0 + C) * vrs, vrs, s.T - 1 - (t0 + C));
        if (sbeta) Dma::beta(sm, bg + (size_t)(t0 + C) * s.H, s.H, s.T - 1 - (t0 + C));
      }

      // ---- update S_e <- gamma^C_e S_e + K^T diag(c_e) U
      f32x4 U[NT];
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) U[rt] = sm.Us[rt][l];
      F Uc[SPW][NT], Ucl[SPW][NT];
#pragma unroll
      for (int i = 0; i < SPW; ++i) {
        const int e = slc(i);
        const float gc = sm.gC[e];
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) S[i][kt] *= gc;
#pragma unroll
        for (int kb = 0; kb < NT; ++kb)
          split_frag(U[kb] * *(const f32x4*)&sm.coef2[e][16 * kb + 4 * g], Uc[i][kb], Ucl[i][kb]);
      }
#pragma unroll
      for (int kb = 0; kb < NT; kb += (NT > 1 ? 2 : 1)) {
        if constexpr (NT > 1) {
          // K^T rows: positions 4 g + j and 16 + 4 g + j of the block pair are
          // adjacent in the operand tile (one 16-byte read per lane)
          Frag8<T> a[KT];
          const int c = key_of_row<C>(16 * kb + 4 * g);
#pragma unroll
          for (int kt = 0; kt < KT; ++kt) a[kt].v = *(const bf16x8*)sm.Kt.at(16 * kt + n, c);
#pragma unroll
          for (int i = 0; i < SPW; ++i) {
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) mma32(S[i][kt], a[kt], Uc[i][kb], Uc[i][kb + 1]);
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) mma32(S[i][kt], a[kt], Ucl[i][kb], Ucl[i][kb + 1]);
          }
        } else {
          F a[KT];
#pragma unroll
          for (int kt = 0; kt < KT; ++kt) a[kt] = ld_frag(sm.Kt.at(16 * kt + n, 4 * g));
#pragma unroll
          for (int i = 0; i < SPW; ++i)
#pragma unroll
            for (int kt = 0; kt < KT; ++kt) {
              mma16(S[i][kt], a[kt], Uc[i][0]);
              mma16(S[i][kt], a[kt], Ucl[i][0]);
            }
        }
      }
      // the next chunk-start state's operand copy, kept in registers for the
      // next W partial and left in shared memory for the output waves
#pragma unroll
      for (int i = 0; i < SPW; ++i)
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
          Sop[i][kt] = cvt_frag<T>(S[i][kt]);
          smd.sop[w * SPW + i][kt][l] = Sop[i][kt];
        }
      // K, Q, a_e and b_e of the next chunk have landed (the Tu, V and beta
      // copies were issued after them)
      if (more) {
        if (sbeta)
          wait_vmcnt<Dma::N_TU + 2>();
        else
          wait_vmcnt<Dma::N_TU + 1>();
      }
    }

    if (s_final) {
#pragma unroll
      for (int i = 0; i < SPW; ++i) {
        const int e = slc(i);
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
          float* dst = s_final + (((size_t)head * E + e) * KD + key_col<KD>(kt, g)) * V + v0 + vc;
#pragma unroll
          for (int j = 0; j < 4; ++j) dst[(size_t)j * V] = S[i][kt][j];
        }
      }
    }
  } else {
    // ================================================= output waves
    const bf16x4 idf = identity_frag();  // for the transposing checkpoint stores
    // Every global store of the forward is issued here.  Under the write
    // traffic of all workgroups a store instruction holds up the wave that
    // issues it for some hundreds of cycles, whatever its size (measured;
    // the state waves would lose the same time), so the stores are 16-byte
    // ones and few (11 per chunk step at E = 8), none in the Q pass (which
    // the state waves wait for at B1), and most between B1 and B2, where the
    // output waves have no other work: checkpoint pieces [0, NB) and the rows
    // of V - W (GDN, while V and the W partials are in shared memory); the
    // other pieces, U and the output rows after B2.
    constexpr int NB = (5 * NPC + 4) / 8;
    const bool rows = w < NT;  // the wave owns row tile w
    for (int ci = 0; ci < nc; ++ci) {
      const int t0 = ci * C;
      const size_t ch = ch0 + ci;
      __syncthreads();  // B0
      if (t0 + C > s.T) zero_tail(t0);

      // ---- the chunk-start state of the wave's slices, then the O partial
      // sum over them of diag(b_e) Q S_e
      F So[SPW][KT];
#pragma unroll
      for (int i = 0; i < SPW; ++i)
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) So[i][kt] = smd.sop[w * SPW + i][kt][l];
      u32x4 ckd[PAIRS ? NPC : 1];  // the pieces' data (filled after B1)
      auto ck_store = [&](int pc) {
        if constexpr (PAIRS) {
          piece_store(ch, pc, ckd[pc]);
        } else {
          const int i = pc / KT, kt = pc % KT;
          T* dst = (T*)sv.Sck + ((ch * E + w * SPW + i) * (size_t)(V / 16) + vt) * KD * 16;
          store_tile16_frag(dst + 256 * kt, So[i][kt], idf, g, n);
        }
      };
      state_pass(sm.Q, So, sm.coef01[1], sm.O[w]);
      __syncthreads();  // B1
      // the checkpoint pieces, read before the state waves replace the copy
      // after B2
      if (PAIRS && train) {
#pragma unroll
        for (int pc = 0; pc < NPC; ++pc) ckd[pc] = piece_read(pc);
      }
      if (train && rows && s.variant == 1) {  // rows of V - W of row tile w, as the state waves form them
        const int rt = w;
        T vr[4];
        f32x4 wq[NG];
#pragma unroll
        for (int j = 0; j < 4; ++j) vr[j] = sm.Vr[16 * rt + 4 * j + g][n];
#pragma unroll
        for (int ww = 0; ww < NG; ++ww) wq[ww] = sm.W[ww][rt][pl];
        f32x4 x;
#pragma unroll
        for (int j = 0; j < 4; ++j) x[j] = Elem<T>::to_f(vr[j]);
#pragma unroll
        for (int ww = 0; ww < NG; ++ww) x -= wq[ww];
        store_tile16(sv.X + ch * C * (size_t)V + (size_t)(16 * rt) * V + v0, x, g, n, V);
      }
      if (train) {
#pragma unroll
        for (int pc = 0; pc < NB; ++pc) ck_store(pc);
      }
      __syncthreads();  // B2

      // ---- O for row tile w: the partials plus M U
      if (w < NT) {
        const int rt = w;
        const int r = 16 * rt + n;
        F mf[NT], ml[NT], Uh[NT], Ul[NT];
        f32x4 U[NT], op[NG];
#pragma unroll
        for (int kb = 0; kb < NT; ++kb) {
          mf[kb] = ld_frag(sm.M.at(r, 16 * kb + 4 * g));
          ml[kb] = ld_frag(sm.ML.at(r, 16 * kb + 4 * g));
          U[kb] = sm.Us[kb][l];
        }
#pragma unroll
        for (int ww = 0; ww < NG; ++ww) op[ww] = sm.O[ww][rt][pl];
        __builtin_amdgcn_sched_barrier(0);  // the reads above stay together
#pragma unroll
        for (int kb = 0; kb < NT; ++kb) split_frag(U[kb], Uh[kb], Ul[kb]);
        f32x4 oacc = zero4();
#pragma unroll
        for (int ww = 0; ww < NG; ++ww) oacc += op[ww];
        mma_k<C>(oacc, [&](int kb) { return mf[kb]; }, [&](int kb) { return Uh[kb]; });
        mma_k<C>(oacc, [&](int kb) { return mf[kb]; }, [&](int kb) { return Ul[kb]; });
        mma_k<C>(oacc, [&](int kb) { return ml[kb]; }, [&](int kb) { return Uh[kb]; });
        if (train) {
#pragma unroll
          for (int pc = NB; pc < NPC; ++pc) ck_store(pc);
          store_tile16(sv.U + ch * C * (size_t)V + (size_t)(16 * rt) * V + v0, U[rt], g, n, V);
        }
        // output rows: lane (g, n) writes row 16 rt + 4 g + n % 4, columns
        // 4 (n / 4) .. + 3
        const f32x4 y = quad_transpose(oacc, n);
        const int t = t0 + 16 * rt + 4 * g + (n & 3);
        if (t < s.T && (!PK || n < 8)) {  // (PK: columns 8..15 repeat 0..7)
          // nontemporal: the tile's rows are whole 32-byte (bf16) or
          // 64-byte pieces that no kernel of the step reads again, and left
          // dirty in L2 their write-back slowed the next kernel
          const size_t off = ((tok0 + t) * s.H + h) * (size_t)V + v0 + 4 * (n >> 2);
          if (s.out_bf16)
            gstore_b64((bf16_t*)out + off, __builtin_bit_cast(u32x2, cvt_frag<bf16_t>(y)));
          else
            gstore_b128((float*)out + off, __builtin_bit_cast(u32x4, y));
        }
      } else if (train) {
#pragma unroll
        for (int pc = NB; pc < NPC; ++pc) ck_store(pc);
      }
    }
  }
}

// ---------------------------------------------------------------- launchers
// Eight waves (two per SIMD) for E = 16, whose state does not fit four waves'
// registers; four waves otherwise (measured faster at E = 8).
template <typename T, int E> constexpr int fwd_waves() { return E >= 16 ? 8 : 4; }

template <typename T, int KD, int C, int E>
static hipError_t prep_inst(const Shape& s, const FwdIn& in, const PrepBufs& p, hipStream_t st) {
  const size_t smem = sizeof(PrepSmem<T, KD, C, E>);
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)k_prep<T, KD, C, E>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    attr_set = true;
  }
  hipLaunchKernelGGL((k_prep<T, KD, C, E>), dim3(s.NH * s.Nc), dim3(prep_waves<E>() * 64), smem, st,
                     s, in, p);
  return hipGetLastError();
}

// The forward with separate state and output waves serves bf16 operands with
// E = 4 or 8 slices; E = 16 (whose state would not fit the registers of four
// waves that share their SIMDs with four more) and fp32 operands (whose tiles
// would not fit the shared memory) keep the single-role kernel.
template <typename T, int KD, int C, int E>
constexpr bool fwd_dual() {
  return sizeof(T) == 2 && E % 4 == 0 && E <= 8 && FwdSmem<T, KD, C, E, 4>::STAGE_Q &&
         sizeof(DualSmem<T, KD, C, E>) <= 160 * 1024;
}

// The same kernel with two slices per tile (inference at E = 16, K = 128,
// chunk 64): 8 value columns per workgroup, twice the workgroups.
template <typename T, int KD, int C, int E>
constexpr bool fwd_pk() {
  return sizeof(T) == 2 && E == 16 && KD == 128 && C == 64 &&
         sizeof(DualSmem<T, KD, C, E, true>) <= 160 * 1024;
}

template <typename T, int KD, int C, int E>
static hipError_t fwd_inst(const Shape& s, const FwdIn& in, const PrepBufs& p, void* o,
                           float* s_final, const SavedBufs* sv, hipStream_t st) {
  SavedBufs none{nullptr, nullptr, nullptr};
  if constexpr (fwd_pk<T, KD, C, E>()) {
    if (!sv) {
      const size_t smem = sizeof(DualSmem<T, KD, C, E, true>);
      static bool attr_pk = false;
      if (!attr_pk) {
        (void)hipFuncSetAttribute((const void*)k_fwd_dual<T, KD, C, E, true>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        attr_pk = true;
      }
      hipLaunchKernelGGL((k_fwd_dual<T, KD, C, E, true>), dim3(s.NH * (s.V / 8)), dim3(512), smem,
                         st, s, in, p, o, s_final, none, 0);
      return hipGetLastError();
    }
  }
  if constexpr (fwd_dual<T, KD, C, E>()) {
    const size_t smem = sizeof(DualSmem<T, KD, C, E>);
    static bool attr_set = false;
    if (!attr_set) {
      (void)hipFuncSetAttribute((const void*)k_fwd_dual<T, KD, C, E>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
      attr_set = true;
    }
    hipLaunchKernelGGL((k_fwd_dual<T, KD, C, E>), dim3(s.NH * (s.V / 16)), dim3(512), smem, st, s,
                       in, p, o, s_final, sv ? *sv : none, sv ? 1 : 0);
    return hipGetLastError();
  }
  constexpr int NW = fwd_waves<T, E>();
  typedef FwdSmem<T, KD, C, E, NW> Sm;
  const size_t smem = sizeof(Sm);
  static bool attr_set = false;
  if (!attr_set) {  // allow more than the default dynamic LDS (best effort)
    (void)hipFuncSetAttribute((const void*)k_fwd<T, KD, C, E, NW>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    attr_set = true;
  }
  hipLaunchKernelGGL((k_fwd<T, KD, C, E, NW>), dim3(s.NH * (s.V / 16)), dim3(NW * 64), smem, st,
                     s, in, p, o, s_final, sv ? *sv : none, sv ? 1 : 0);
  return hipGetLastError();
}

#define TLA_DISPATCH(KD_, C_, E_, CALL)                          \
  if (s.K == KD_ && s.C == C_ && s.E == E_) {                    \
    if (s.in_bf16) return CALL(bf16_t, KD_, C_, E_);             \
    return CALL(float, KD_, C_, E_);                             \
  }

#define TLA_FOR_EACH_INSTANCE(CALL) \
  TLA_DISPATCH(16, 16, 1, CALL)     \
  TLA_DISPATCH(16, 16, 2, CALL)     \
  TLA_DISPATCH(16, 16, 4, CALL)     \
  TLA_DISPATCH(16, 16, 8, CALL)     \
  TLA_DISPATCH(16, 16, 16, CALL)    \
  TLA_DISPATCH(32, 32, 4, CALL)     \
  TLA_DISPATCH(64, 32, 8, CALL)     \
  TLA_DISPATCH(64, 64, 16, CALL)     \
  TLA_DISPATCH(32, 32, 32, CALL)     \
  TLA_DISPATCH(128, 64, 1, CALL)    \
  TLA_DISPATCH(128, 64, 4, CALL)    \
  TLA_DISPATCH(128, 64, 8, CALL)    \
  TLA_DISPATCH(128, 64, 16, CALL)   \
  TLA_DISPATCH(128, 32, 8, CALL)

hipError_t launch_prep(const Shape& s, const FwdIn& in, const PrepBufs& p, hipStream_t st) {
#define CALL_PREP(T_, KD_, C_, E_) prep_inst<T_, KD_, C_, E_>(s, in, p, st)
  TLA_FOR_EACH_INSTANCE(CALL_PREP)
#undef CALL_PREP
  return hipErrorInvalidValue;
}

hipError_t launch_fwd(const Shape& s, const FwdIn& in, const PrepBufs& p, void* o, float* s_final,
                      const SavedBufs* saved, hipStream_t st) {
#define CALL_FWD(T_, KD_, C_, E_) fwd_inst<T_, KD_, C_, E_>(s, in, p, o, s_final, saved, st)
  TLA_FOR_EACH_INSTANCE(CALL_FWD)
#undef CALL_FWD
  return hipErrorInvalidValue;
}

template <typename T, int KD, int C, int E>
static bool fits_inst() {
  return sizeof(FwdSmem<T, KD, C, E, fwd_waves<T, E>()>) <= 160 * 1024 &&
         sizeof(PrepSmem<T, KD, C, E>) <= 160 * 1024;
}

bool fits_lds(int K, int C, int E, bool bf16) {
#define FITS(T_, KD_, C_, E_) fits_inst<T_, KD_, C_, E_>()
  const tla::Shape s{0, 1, 1, 1, K, 16, E, C, 1, 1, bf16 ? 1 : 0, 0, 0};
  TLA_FOR_EACH_INSTANCE(FITS)
#undef FITS
  return false;
}

bool have_instance(int K, int C, int E) {
  return (K == 16 && C == 16 && (E == 1 || E == 2 || E == 4 || E == 8 || E == 16)) ||
         (K == 32 && C == 32 && E == 4) ||
         (K == 32 && C == 32 && E == 32) || (K == 64 && C == 32 && E == 8) ||
         (K == 64 && C == 64 && E == 16) ||
         (K == 128 && C == 64 && (E == 1 || E == 4 || E == 8 || E == 16)) ||
         (K == 128 && C == 32 && E == 8);
}

}  // namespace tla
