// Backward of chunkwise triadic linear attention on gfx950.
//
// The structure follows the paper's backward (Appendix A, "Kernels"): a
// short reverse recurrence over chunks produces the gradient of every
// chunk-end state, after which every other gradient is computed for all
// chunks in parallel, with fixed-order reductions and no atomics.  The chunk
// equations are the reverse-mode derivative of Eq. joint-chunk (with
// Eq. joint-gram / joint-solve) and are restated per kernel below.  With
// N = I + L, Tu = N^{-1} diag(beta), A_hat = A_kk o R, and dS'_e the gradient
// of the state at the end of the chunk:
//
//   k_bwd_rec   (head, 16-column value tile), chunks in reverse:
//     dU   = M^T dO + sum_e diag(c_e) K dS'_e
//     dW   = -Tu^T dU                        (GDN; sGLA has no W)
//     dS_e = gamma^C_e dS'_e + Q^T diag(b_e) dO + K^T diag(a_e) dW
//   k_bwd_state (head, chunk):
//     X_e = dO S_e^T, Y_e = dW S_e^T, V'_e = U dS'_e^T
//     dq_s = sum_e diag(b_e) X_e;  dk_s = sum_e diag(a_e) Y_e + diag(c_e) V'_e
//     db_e = rowsum(Q o X_e), da_e = rowsum(K o Y_e), dc_e = rowsum(K o V'_e)
//     dgamma^C_e = <S_e, dS'_e>
//   k_bwd_chunk (head, chunk):
//     dM = dO U^T (lower incl. diagonal); dA_qk = dM o R'; dR' = dM o A_qk
//     GDN: dTu = dU (V - W)^T; P = N^{-T} dTu; dbeta_r = P_rr + sum_s dL_rs A_hat_rs
//          dL = tril(-P Tu^T, -1); dA_hat = diag(beta) dL
//          dA_kk = dA_hat o R; dR = dA_hat o A_kk; dv = Tu^T dU = -dW
//     sGLA: dv = diag(beta) dU; dbeta_r = <dU_r, v_r>
//     dq = dq_s + dA_qk K;  dk = dk_s + dA_qk^T Q + (dA_kk + dA_kk^T) K
//     R, R' (Eq. joint-gram):  phi_e[r,s] = (dR'[r,s] q2_r[e] + dR[r,s] k2_r[e]) k2_s[e] Gamma_e[r,s]
//          dq2_r[e] += sum_s dR'[r,s] k2_s[e] Gamma_e;  dk2_s[e] += sum_r (dR' q2_r + dR k2_r) Gamma_e
//          dk2_r[e] += sum_s dR[r,s] k2_s[e] Gamma_e;   dG_r[e] += sum_s phi;  dG_s[e] -= sum_r phi
//     coefficient vectors: dk2 += da o gamma + dc o gamma^C/gamma;  dq2 += db o gamma
//          dG += da o a + db o b - dc o c;  dG_C += sum_r dc c + gamma^C dgamma^C
//     dg_j = sum_{r >= j in the chunk} dG_r   (G is the in-chunk cumulative log-gate)
#include <type_traits>

#include "tla_common.hpp"
#include "tla_internal.hpp"

namespace tla {

template <typename T>
__device__ __forceinline__ void bcopy8(T* dst, const T* src) {
  if constexpr (sizeof(T) == 2) {
    *(uint4*)dst = *(const uint4*)src;
  } else {
    ((float4*)dst)[0] = ((const float4*)src)[0];
    ((float4*)dst)[1] = ((const float4*)src)[1];
  }
}
template <typename T>
__device__ __forceinline__ void bzero8(T* dst) {
  if constexpr (sizeof(T) == 2) {
    *(uint4*)dst = make_uint4(0, 0, 0, 0);
  } else {
    ((float4*)dst)[0] = make_float4(0, 0, 0, 0);
    ((float4*)dst)[1] = make_float4(0, 0, 0, 0);
  }
}

// Gradients are written in the call's output type (fp32 or bf16).
__device__ __forceinline__ void store_out(void* base, size_t off, float x, int out_bf16) {
  if (out_bf16)
    ((bf16_t*)base)[off] = Elem<bf16_t>::from_f(x);
  else
    ((float*)base)[off] = x;
}

// Rows i .. i + 3 of column c of a row-major shared-memory tile, p =
// &tile[i][c] with a row pitch of P elements: the fragment that row c of the
// transposed tile would give at columns i .. i + 3.
template <int P>
__device__ __forceinline__ f32x4 col_frag(const float* p) {
  return f32x4{p[0], p[P], p[2 * P], p[3 * P]};
}
template <int P>
__device__ __forceinline__ bf16x4 col_frag(const bf16_t* p) {
  const uint32_t a = (uint32_t)p[0] | ((uint32_t)p[P] << 16);
  const uint32_t b = (uint32_t)p[2 * P] | ((uint32_t)p[3 * P] << 16);
  return __builtin_bit_cast(bf16x4, make_uint2(a, b));
}

template <int D, typename FA, typename FB>
__device__ __forceinline__ void bmma_k(f32x4& acc, FA fa, FB fb) {
  constexpr int NB = D / 16;
#pragma unroll
  for (int kb = 0; kb + 1 < NB; kb += 2) mma32(acc, fa(kb), fa(kb + 1), fb(kb), fb(kb + 1));
  if constexpr (NB & 1) mma16(acc, fa(NB - 1), fb(NB - 1));
}

template <int E> constexpr int bwd_waves() { return E >= 8 ? 8 : 4; }

// ============================================================ reverse recurrence
template <typename T, int KD, int C, int E, int NW>
struct RecSmem {
  static constexpr int KP = KD + 8;  // 16-byte rows: 32-deep A operands are one 16-byte read
  static constexpr int CP = C + 4;
  static constexpr int NT = C / 16;
  static constexpr int E4 = (E + 3) & ~3;
  static constexpr bool SPLIT = sizeof(T) == 2;
  // rows of K (A operand of K dS'); fp32 operands read them from global memory
  // so that the fp32 plan fits the 160 KiB of LDS
  static constexpr bool STAGE_K = sizeof(T) == 2;
  alignas(16) T K[STAGE_K ? C : 1][KP];
  alignas(16) T Kt[KD][CP];      // K^T
  alignas(16) T Qt[KD][CP];      // Q^T
  alignas(16) T dOt[16][CP];     // dO tile, transposed
  // M and Tu row-major (hi; lo below): the A operands of M^T dO and Tu^T dU
  // are read down their columns
  alignas(16) T M[C][CP];
  alignas(16) T Tu[C][CP];
  alignas(16) T ML[SPLIT ? C : 1][CP];
  alignas(16) T TuL[SPLIT ? C : 1][CP];
  alignas(16) float coef[3][E][C];
  alignas(16) float gC[E4];
  alignas(16) f32x4 X[NW][NT][64];  // per-wave partials of sum_e diag(c_e) K dS'_e
  alignas(16) typename Elem<T>::frag dUs[SPLIT ? 2 : 1][NT][64];  // dU as B operands (hi, lo)
  alignas(16) f32x4 dWs[NT][64];
  alignas(16) f32x4 dUf[NT][64];  // fp32 dU, stored to global memory at the next step
};

// Register staging of one chunk's inputs for the reverse recurrence: the
// global loads for chunk ci - 1 are issued while chunk ci is computed, and
// copied to shared memory at the top of the next step.  K^T, Q^T, M and Tu
// arrive from the prep kernel already in operand layout and split, so only the
// dO tile is transposed here.  Loads are unconditional (rows past T read a
// clamped row and are zeroed when stored) and waves past the last piece of a
// loop step skip it (a scalar branch).
template <typename T, int KD, int C, int E, int NTHR>
struct RecStage {
  typedef OpTiles<T, KD, C> OT;
  static constexpr int EC = 16 / (int)sizeof(T);        // elements per 16-byte chunk
  static constexpr int NRC = C * KD / EC;                // chunks of the K rows
  static constexpr int NTC = 2 * KD * C / EC;            // chunks of K^T and Q^T
  static constexpr int NMC = 2 * OT::NS * C * C / EC;    // chunks of M and Tu (hi, lo)
  static constexpr int RB = C / 4;
  static constexpr int NR = (NRC + NTHR - 1) / NTHR;
  static constexpr int NTT = (NTC + NTHR - 1) / NTHR;
  static constexpr int NM = (NMC + NTHR - 1) / NTHR;
  static constexpr int NDB = (RB * 4 + NTHR - 1) / NTHR;       // 4 x 4 blocks of the dO tile
  static constexpr int NCB = (3 * E * C / 4 + NTHR - 1) / NTHR;
  static constexpr int E4 = (E + 3) & ~3;
  static constexpr int DW = sizeof(T) == 2 ? 2 : 4;            // words per 4 elements
  static constexpr bool ROWS = sizeof(T) == 2;                 // K rows staged (bf16 only)
  uint4 k[ROWS ? NR : 1], tt[NTT], mt[NM];
  uint32_t d[NDB][4][DW];
  f32x4 c[NCB];
  float gc;

  // parts: 1 = the K rows, K^T, Q^T and the dO tile; 2 = M, Tu and the
  // vectors (the two halves are issued at different points of a chunk step)
  __device__ __forceinline__ void load(const Shape& s, const PrepBufs& p, const T* Kg,
                                       const T* Qg, const T* dOg, size_t ch, int ci,
                                       int parts = 3) {
    const int tid = threadIdx.x;
    const int w0 = 64 * wave_id();  // first thread of this wave (wave-uniform)
    const int t0 = ci * C;
    const size_t krs = (size_t)s.H * KD, vrs = (size_t)s.H * s.V;
    const T* ops = (const T*)p.ops + ch * OT::STRIDE;
    if (parts & 1) {
      if constexpr (ROWS) {
#pragma unroll
        for (int i = 0; i < NR; ++i) {
          if (w0 + i * NTHR >= NRC) continue;
          const int idx = min(tid + i * NTHR, NRC - 1);
          const int r = idx / (KD / EC), c0 = EC * (idx % (KD / EC));
          k[i] = *(const uint4*)(Kg + (size_t)min(t0 + r, s.T - 1) * krs + c0);
        }
      }
#pragma unroll
      for (int i = 0; i < NTT; ++i) {
        if (w0 + i * NTHR >= NTC) continue;
        tt[i] = ((const uint4*)(ops + OT::Kt))[min(tid + i * NTHR, NTC - 1)];
      }
#pragma unroll
      for (int i = 0; i < NDB; ++i) {
        if (w0 + i * NTHR >= RB * 4) continue;
        const int blk = min(tid + i * NTHR, RB * 4 - 1);
        const int rb = blk % RB, c4 = blk / RB;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int t = min(t0 + 4 * rb + rr, s.T - 1);
          ld_words(d[i][rr], dOg + (size_t)t * vrs + 4 * c4);
        }
      }
    }
    if (!(parts & 2)) return;
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      if (w0 + i * NTHR >= NMC) continue;
      mt[i] = ((const uint4*)(ops + OT::M))[min(tid + i * NTHR, NMC - 1)];
    }
    const float* cg = p.coef + ch * 3 * E * C;
#pragma unroll
    for (int i = 0; i < NCB; ++i)
      if (w0 + i * NTHR < 3 * E * C / 4)
        c[i] = *(const f32x4*)(cg + 4 * min(tid + i * NTHR, 3 * E * C / 4 - 1));
    gc = p.gC[ch * E4 + min(tid, E4 - 1)];
  }

  template <typename Sm>
  __device__ __forceinline__ void store(Sm& sm, int variant, int t0, int nT,
                                        int parts = 3) const {
    const int tid = threadIdx.x;
    if (parts & 1) {
    if constexpr (ROWS) {
#pragma unroll
      for (int i = 0; i < NR; ++i) {
        const int idx = tid + i * NTHR;
        if (idx >= NRC) continue;
        const int r = idx / (KD / EC), c0 = EC * (idx % (KD / EC));
        lds_put16(&sm.K[r][c0], (t0 + r < nT) ? k[i] : make_uint4(0, 0, 0, 0));
      }
    }
    // K^T then Q^T (rows past T are already zero)
    constexpr int PERT = KD * C / EC;
#pragma unroll
    for (int i = 0; i < NTT; ++i) {
      const int idx = tid + i * NTHR;
      if (idx >= NTC) continue;
      const int mtx = idx / PERT, j = idx % PERT;
      const int r = j / (C / EC), c0 = EC * (j % (C / EC));
      lds_put16(mtx ? &sm.Qt[r][c0] : &sm.Kt[r][c0], tt[i]);
    }
#pragma unroll
    for (int i = 0; i < NDB; ++i) {
      const int blk = tid + i * NTHR;
      const int rb = blk % RB, c4 = blk / RB;
      if (blk < RB * 4) {
        uint32_t dd[4][DW];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const bool ok = t0 + 4 * rb + rr < nT;
#pragma unroll
          for (int j = 0; j < DW; ++j) dd[rr][j] = ok ? d[i][rr][j] : 0u;
        }
#pragma unroll
        for (int cc = 0; cc < 4; ++cc)
          lds_put4(&sm.dOt[4 * c4 + cc][4 * rb], word_elem<T>(dd[0], cc), word_elem<T>(dd[1], cc),
                   word_elem<T>(dd[2], cc), word_elem<T>(dd[3], cc));
      }
    }
    }
    if (!(parts & 2)) return;
    // M and Tu chunks: matrix m (M hi, lo, Tu hi, lo for bf16; M, Tu for fp32)
    constexpr int PER = C * C / EC;
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      const int idx = tid + i * NTHR;
      if (idx >= NMC) continue;
      const int mtx = idx / PER, j = idx % PER;
      const int r = j / (C / EC), c0 = EC * (j % (C / EC));
      T* dst;
      if constexpr (OT::NS == 2)
        dst = (mtx == 0) ? &sm.M[r][c0] : (mtx == 1) ? &sm.ML[r][c0] : (mtx == 2) ? &sm.Tu[r][c0] : &sm.TuL[r][c0];
      else
        dst = (mtx == 0) ? &sm.M[r][c0] : &sm.Tu[r][c0];
      lds_put16(dst, mt[i]);
    }
    float* cs = &sm.coef[0][0][0];
#pragma unroll
    for (int i = 0; i < NCB; ++i) {
      const int idx = tid + i * NTHR;
      if (idx < 3 * E * C / 4) *(f32x4*)(cs + 4 * idx) = c[i];
    }
    if (tid < E4) sm.gC[tid] = gc;
  }
};

// PDS (bf16 operands with a final-state gradient): the chunk-end state
// gradients dS' enter K dS'_e as bf16 (hi, lo) pairs and are stored as two
// bf16 tiles (dSck, dSck_lo).  A given final-state gradient makes dS' of the
// last chunks far larger than elsewhere in the sequence, and one bf16
// rounding of it would then dominate the gradients of those chunks.
template <typename T, int KD, int C, int E, int NW, bool PDS>
__global__ __launch_bounds__(NW * 64) void k_bwd_rec(Shape s, FwdIn in, const void* dOv,
                                                     const float* dS_final, PrepBufs p,
                                                     BwdBufs bb, float* ds0) {
  constexpr int SPW = (E + NW - 1) / NW;
  constexpr bool RAGGED = E % NW != 0;  // some waves own fewer slices
  constexpr int NT = C / 16;
  constexpr int KT = KD / 16;
  constexpr int NTHR = NW * 64;
  typedef typename Elem<T>::frag F;
  typedef RecSmem<T, KD, C, E, NW> Sm;
  // eight-wave instances (E = 16) have half the registers per lane: they load
  // each chunk's inputs at its own start instead of one chunk ahead, and
  // reuse operand fragments over fewer slices at a time
  constexpr bool PREFETCH = SPW == 1 || NW <= 4;
  // the Tu^T operand of dW, gathered from the columns of the staged Tu, is
  // read while dU is formed (instances with registers to spare)
  constexpr bool EARLY_T = PREFETCH && !PDS;
  constexpr int NKB = C / 16;
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

  // dS[i][kt] = dS_e[16 kt + 4 g + j][v0 + n], e = w * SPW + i
  f32x4 dS[SPW][KT];
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const int e = w * SPW + i;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      f32x4 x = zero4();
      if (dS_final && e < E) {
        const float* src = dS_final + (((size_t)head * E + e) * KD + key_col<KD>(kt, g)) * V + v0 + n;
#pragma unroll
        for (int j = 0; j < 4; ++j) x[j] = src[(size_t)j * V];
      }
      dS[i][kt] = x;
    }
  }

  const T* Kg = (const T*)in.k + (tok0 * s.H + h) * KD;
  const T* Qg = (const T*)in.q + (tok0 * s.H + h) * KD;
  const T* dOg = (const T*)dOv + (tok0 * s.H + h) * (size_t)V + v0;
  const size_t krs = (size_t)s.H * KD;

  const bf16x4 idf = identity_frag();  // for the transposing dS' stores
  // row tile w of dU and dW of chunk ch (from their shared-memory copies)
  auto store_dudw = [&](size_t chs) {
    if (w < NT) {
      const int rt = w;
      store_tile16(bb.dU + chs * C * (size_t)V + (size_t)(16 * rt) * V + v0, sm.dUf[rt][l], g, n, V);
      store_tile16(bb.dW + chs * C * (size_t)V + (size_t)(16 * rt) * V + v0,
                   s.variant == 1 ? sm.dWs[rt][l] : zero4(), g, n, V);
    }
  };
  RecStage<T, KD, C, E, NTHR> stage;
  if constexpr (PREFETCH)
    if (nc > 0) stage.load(s, p, Kg, Qg, dOg, (size_t)head * s.Nc + nc - 1, nc - 1);
  for (int ci = nc - 1; ci >= 0; --ci) {
    const int t0 = ci * C;
    const size_t ch = (size_t)head * s.Nc + ci;
    __syncthreads();
    // ---- this chunk's inputs to LDS; the next chunk's loads go in flight
    if constexpr (PREFETCH) {
      stage.store(sm, s.variant, t0, s.T);
    } else {
#pragma unroll
      for (int part = 1; part <= 2; ++part) {  // in halves: fewer live registers
        RecStage<T, KD, C, E, NTHR> now;
        now.load(s, p, Kg, Qg, dOg, ch, ci, part);
        now.store(sm, s.variant, t0, s.T, part);
      }
    }
    // the previous chunk's dU and dW leave now: stored where they are formed,
    // they would precede the prefetch loads that the staging above waits for,
    // and a wave's wait for loads also waits for its earlier stores
    if (ci + 1 < nc) store_dudw(ch + 1);
    __syncthreads();

    // ---- operand copies of dS' (gradient of the chunk-end state), stored for
    // the chunk-parallel kernel
    F dSop[SPW][KT], dSlo[PDS ? SPW : 1][PDS ? KT : 1];
#pragma unroll
    for (int i = 0; i < SPW; ++i)
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        dSop[i][kt] = cvt_frag<T>(dS[i][kt]);
        if constexpr (PDS) dSlo[i][kt] = cvt_frag<T>(dS[i][kt] - frag_to_f(dSop[i][kt]));
      }
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int e = w * SPW + i;
      if (RAGGED && e >= E) continue;
      const size_t toff = ((ch * E + e) * (size_t)(V / 16) + vt) * KD * 16;
      T* dst = (T*)bb.dSck + toff;
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        if constexpr (sizeof(T) == 2) {
          store_tile16_frag(dst + 256 * kt, dSop[i][kt], idf, g, n);
          if constexpr (PDS) store_tile16_frag((T*)bb.dSck_lo + toff + 256 * kt, dSlo[i][kt], idf, g, n);
        } else {
          store_tile16(dst + 256 * kt, dS[i][kt], g, n);
        }
      }
    }

    // ---- partial of sum_e diag(c_e) K dS'_e over the owned slices
    // (K fragments are read once per key block and reused for every owned slice)
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) {
      const int r = 16 * rt + n;
      const bool kok = t0 + r < s.T;
      const T* krow = Kg + (size_t)(kok ? t0 + r : 0) * krs;
      auto kfrag = [&](int kb) -> F {
        if constexpr (Sm::STAGE_K) return ld_frag(&sm.K[r][key_col<KD>(kb, g)]);
        else return kok ? ld_frag(krow + key_col<KD>(kb, g)) : cvt_frag<T>(zero4());
      };
      // keys key_col(kb, g) .. + 7 of the row (kb even): one 32-deep A operand
      auto kfrag8 = [&](int kb) -> Frag8<T> {
        const int c = key_col<KD>(kb, g);
        Frag8<T> f;
        if constexpr (sizeof(T) == 2) {
          if constexpr (Sm::STAGE_K) {
            f.v = *(const bf16x8*)&sm.K[r][c];
          } else {
            const uint4 x = kok ? *(const uint4*)(krow + c) : make_uint4(0, 0, 0, 0);
            f.v = __builtin_bit_cast(bf16x8, x);
          }
        } else {
          f.lo = frag_to_f(kfrag(kb));
          f.hi = kok ? ld_frag(krow + c + 4) : zero4();
          if constexpr (Sm::STAGE_K) f.hi = ld_frag(&sm.K[r][c + 4]);
        }
        return f;
      };
      constexpr int GZ = PREFETCH ? SPW : 1;  // slices per pass over the K fragments
      f32x4 z[SPW];
#pragma unroll
      for (int i = 0; i < SPW; ++i) z[i] = zero4();
#pragma unroll
      for (int i0 = 0; i0 < SPW; i0 += GZ) {
#pragma unroll
        for (int kb = 0; kb + 1 < KT; kb += 2) {
          const Frag8<T> kk = kfrag8(kb);
#pragma unroll
          for (int i = i0; i < i0 + GZ; ++i)
            if (!RAGGED || w * SPW + i < E) {
              mma32(z[i], kk, dSop[i][kb], dSop[i][kb + 1]);
              if constexpr (PDS) mma32(z[i], kk, dSlo[i][kb], dSlo[i][kb + 1]);
            }
        }
        if constexpr (KT & 1) {
          const F k0 = kfrag(KT - 1);
#pragma unroll
          for (int i = i0; i < i0 + GZ; ++i)
            if (!RAGGED || w * SPW + i < E) {
              mma16(z[i], k0, dSop[i][KT - 1]);
              if constexpr (PDS) mma16(z[i], k0, dSlo[i][KT - 1]);
            }
        }
      }
      f32x4 acc = zero4();
#pragma unroll
      for (int i = 0; i < SPW; ++i) {
        const int e = w * SPW + i;
        if (!RAGGED || e < E) acc += *(const f32x4*)&sm.coef[2][e][16 * rt + 4 * g] * z[i];
      }
      sm.X[w][rt][l] = acc;
    }
    __syncthreads();

    // the next chunk's rows are in flight while this chunk computes
    if constexpr (PREFETCH)
      if (ci > 0) stage.load(s, p, Kg, Qg, dOg, ch - 1, ci - 1, 1);
    // ---- dU = M^T dO + sum of the partials, then dW = -Tu^T dU: wave w < NT
    // forms row tile w of each, and the tiles are exchanged through LDS
    F tuf[2][NKB];
    if (w < NT) {
      const int rt = w;
      const int r = 16 * rt + n;
      if constexpr (EARLY_T) {  // Tu^T fragments for dW below, read under dU
        if (s.variant == 1) {
#pragma unroll
          for (int kb = 0; kb < NKB; ++kb) {
            tuf[0][kb] = col_frag<Sm::CP>(&sm.Tu[16 * kb + 4 * g][r]);
            if constexpr (Sm::SPLIT) tuf[1][kb] = col_frag<Sm::CP>(&sm.TuL[16 * kb + 4 * g][r]);
          }
        }
      }
      f32x4 acc = zero4();
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) acc += sm.X[ww][rt][l];
      auto dof = [&](int kb) { return ld_frag(&sm.dOt[n][16 * kb + 4 * g]); };
      bmma_k<C>(acc, [&](int kb) { return col_frag<Sm::CP>(&sm.M[16 * kb + 4 * g][r]); }, dof);
      if constexpr (Sm::SPLIT)
        bmma_k<C>(acc, [&](int kb) { return col_frag<Sm::CP>(&sm.ML[16 * kb + 4 * g][r]); }, dof);
      F hi, lo;
      split_frag(acc, hi, lo);
      sm.dUs[0][rt][l] = hi;
      if constexpr (Sm::SPLIT) sm.dUs[1][rt][l] = lo;
      sm.dUf[rt][l] = acc;
    }
    __syncthreads();
    if (w < NT) {
      const int rt = w;
      f32x4 acc = zero4();
      if (s.variant == 1) {
        const int r = 16 * rt + n;
        auto tfr = [&](int part, int kb) -> F {
          if constexpr (EARLY_T) return tuf[part][kb];
          else return col_frag<Sm::CP>(part ? &sm.TuL[16 * kb + 4 * g][r] : &sm.Tu[16 * kb + 4 * g][r]);
        };
        auto th = [&](int kb) { return tfr(0, kb); };
        bmma_k<C>(acc, th, [&](int kb) { return sm.dUs[0][kb][l]; });
        if constexpr (Sm::SPLIT) {
          bmma_k<C>(acc, th, [&](int kb) { return sm.dUs[1][kb][l]; });
          bmma_k<C>(acc, [&](int kb) { return tfr(1, kb); },
                    [&](int kb) { return sm.dUs[0][kb][l]; });
        }
        acc = -acc;
        sm.dWs[rt][l] = acc;
      }
    }
    f32x4 dW[NT];
    if (s.variant == 1) {
      __syncthreads();
#pragma unroll
      for (int kb = 0; kb < NT; ++kb) dW[kb] = sm.dWs[kb][l];
    } else {
#pragma unroll
      for (int kb = 0; kb < NT; ++kb) dW[kb] = zero4();
    }

    // (the next chunk's M, Tu and vectors; the update below reads its
    // coefficients from LDS)
    if constexpr (PREFETCH)
      if (ci > 0) stage.load(s, p, Kg, Qg, dOg, ch - 1, ci - 1, 2);
    // ---- dS_e <- gamma^C_e dS'_e + Q^T diag(b_e) dO + K^T diag(a_e) dW
    // (B operands of a group of owned slices first; each Q^T / K^T fragment is
    // read once per group, one key tile ahead of its MFMAs; four-wave
    // instances take all owned slices at once).  The variant is a constant
    // inside: no branch splits the loop.  Operands: diag(b_e) dO enters as a
    // bf16 (hi, lo) pair; diag(a_e) dW as one bf16 rounding (its low part
    // moves the gradients by less than a tenth of the bf16 parity bound, the
    // high part alone of diag(b_e) dO puts dv past it), except in the
    // instances for a given final-state gradient, which keep both parts.
    constexpr int GS = PREFETCH ? SPW : 1;
    constexpr bool DW_LO = Sm::SPLIT && PDS;
    auto update = [&](auto gdn_c) {
      constexpr bool GDN = decltype(gdn_c)::value;
#pragma unroll
      for (int i0 = 0; i0 < SPW; i0 += GS) {
        F bh[GS][NT], bl[GS][NT], ah[GS][NT], al[GS][NT];
        float gcs[GS];
#pragma unroll
        for (int ii = 0; ii < GS; ++ii) {
          const int e = w * SPW + i0 + ii;
          if (RAGGED && e >= E) continue;
          gcs[ii] = sm.gC[e];
#pragma unroll
          for (int kb = 0; kb < NT; ++kb) {
            const f32x4 dov = ld4_f(&sm.dOt[n][16 * kb + 4 * g]);
            split_frag(dov * *(const f32x4*)&sm.coef[1][e][16 * kb + 4 * g], bh[ii][kb], bl[ii][kb]);
            if constexpr (GDN)
              split_frag(dW[kb] * *(const f32x4*)&sm.coef[0][e][16 * kb + 4 * g], ah[ii][kb],
                         al[ii][kb]);
          }
        }
        // Q^T / K^T rows: positions 4 g + j and 16 + 4 g + j of a block pair
        // are adjacent in the operand tiles (position r at column
        // key_of_row(r)); element kb of a row's fragments is the 16-deep half
        // kb % 2 of the pair kb / 2
        F qf[2][NT], kf[2][NT];
        auto load_kt = [&](int kt, F(&q)[NT], F(&k)[NT]) {
          const int r = 16 * kt + n;
#pragma unroll
          for (int kb = 0; kb < NT; ++kb) {
            const int c = key_of_row<C>(16 * (kb & ~1) + 4 * g) + (NT > 1 ? 4 * (kb & 1) : 0);
            q[kb] = ld_frag(&sm.Qt[r][c]);
            if constexpr (GDN) k[kb] = ld_frag(&sm.Kt[r][c]);
          }
        };
        load_kt(0, qf[0], kf[0]);
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
          if (kt + 1 < KT) load_kt(kt + 1, qf[(kt + 1) & 1], kf[(kt + 1) & 1]);
          const F* q = qf[kt & 1];
          const F* k = kf[kt & 1];
          f32x4 acc[GS];
#pragma unroll
          for (int ii = 0; ii < GS; ++ii) acc[ii] = dS[i0 + ii][kt] * gcs[ii];
#pragma unroll
          for (int kb = 0; kb + 1 < NT; kb += 2) {
#pragma unroll
            for (int ii = 0; ii < GS; ++ii) {
              if (RAGGED && w * SPW + i0 + ii >= E) continue;
              mma32(acc[ii], q[kb], q[kb + 1], bh[ii][kb], bh[ii][kb + 1]);
              if constexpr (Sm::SPLIT) mma32(acc[ii], q[kb], q[kb + 1], bl[ii][kb], bl[ii][kb + 1]);
              if constexpr (GDN) {
                mma32(acc[ii], k[kb], k[kb + 1], ah[ii][kb], ah[ii][kb + 1]);
                if constexpr (DW_LO) mma32(acc[ii], k[kb], k[kb + 1], al[ii][kb], al[ii][kb + 1]);
              }
            }
          }
          if constexpr (NT & 1) {
            const int kb = NT - 1;
#pragma unroll
            for (int ii = 0; ii < GS; ++ii) {
              if (RAGGED && w * SPW + i0 + ii >= E) continue;
              mma16(acc[ii], q[kb], bh[ii][kb]);
              if constexpr (Sm::SPLIT) mma16(acc[ii], q[kb], bl[ii][kb]);
              if constexpr (GDN) {
                mma16(acc[ii], k[kb], ah[ii][kb]);
                if constexpr (DW_LO) mma16(acc[ii], k[kb], al[ii][kb]);
              }
            }
          }
#pragma unroll
          for (int ii = 0; ii < GS; ++ii)
            if (!RAGGED || w * SPW + i0 + ii < E) dS[i0 + ii][kt] = acc[ii];
        }
      }
    };
    if (s.variant == 1)
      update(std::integral_constant<bool, true>{});
    else
      update(std::integral_constant<bool, false>{});
  }
  if (nc > 0) store_dudw((size_t)head * s.Nc);  // chunk 0 (its copies are unchanged since)

  if (ds0) {
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int e = w * SPW + i;
      if (RAGGED && e >= E) continue;
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        float* dst = ds0 + (((size_t)head * E + e) * KD + key_col<KD>(kt, g)) * V + v0 + n;
#pragma unroll
        for (int j = 0; j < 4; ++j) dst[(size_t)j * V] = dS[i][kt][j];
      }
    }
  }
}

// ===================================================== state-gradient contractions
// One workgroup per (head, chunk) with eight waves (two per SIMD).  Wave w
// owns the key columns of quarter q = w % 4 ([16 CTW q, 16 CTW (q + 1))) and
// the row tiles of half w / 4.  The chunk's dO, dW and U rows (A operands;
// dW and U as bf16 hi + lo pairs) are staged in LDS once; the chunk-start
// state S_e and the chunk-end state gradient dS'_e stream from their tiled
// stores as B operands of 32-deep MFMAs over pairs of 16-column value blocks,
// each pair reloaded for the next slice as soon as this slice is done with it
// (the two row halves load the same B data; the second request hits the
// cache).  The rows of Q and K that the row sums need live in registers.
constexpr int STATE_NW = 8;
constexpr int STATE_NTHR = STATE_NW * 64;

template <typename T, int KD, int C, int E>
struct StateSmem {
  static constexpr bool SPLIT = sizeof(T) == 2;
  // fp32 instances stage one 32-column pair of value blocks at a time (LDS budget)
  static constexpr bool STAGE_ALL = sizeof(T) == 2;
  static constexpr int NCOL = STAGE_ALL ? 128 : 32;    // staged columns (V <= 128)
  static constexpr int VS = NCOL + (SPLIT ? 8 : 4);     // row stride, conflict-free b128 reads
  alignas(16) T dO[C][VS];
  alignas(16) T dWh[C][VS], Uh[C][VS];
  alignas(16) T dWl[SPLIT ? C : 1][VS], Ul[SPLIT ? C : 1][VS];
  alignas(16) float coef[3][E][C];
  alignas(16) float red[2][4][3][C];  // per key quarter row-sum partials, by slice parity
  alignas(16) float dcf[3][E][C];
  alignas(16) float gred[4][E];
};

// PDS: the chunk-end state gradients arrive as bf16 (hi, lo) tile pairs
// (see k_bwd_rec) and enter U dS'^T and <S, dS'> with both parts.
template <typename T, int KD, int C, int E, bool PDS>
__global__ __launch_bounds__(STATE_NTHR) void k_bwd_state(Shape s, FwdIn in, const void* dOv,
                                                          PrepBufs p, SavedBufs sv, BwdBufs bb) {
  constexpr int NT = C / 16;
  constexpr int KT = KD / 16;
  constexpr int CTW = (KT + 3) / 4;      // key column tiles per wave
  constexpr int RTW = NT > 1 ? NT / 2 : 1;  // row tiles per wave
  constexpr int E4 = (E + 3) & ~3;
  constexpr int NPMAX = 4;               // pairs of value blocks, V <= 128
  constexpr int NTHR = STATE_NTHR;
  typedef StateSmem<T, KD, C, E> Sm;
  constexpr bool SPLIT = Sm::SPLIT;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Sm& sm = *reinterpret_cast<Sm*>(smem_raw);

  const int tid = threadIdx.x, w = wave_id(), l = lane_id(), g = l >> 4, n = l & 15;
  const int q = w & 3;                   // key quarter
  const int rt0 = (w >> 2) * RTW;        // first owned row tile (>= NT: no rows)
  const bool rows = rt0 < NT;
  const int V = s.V;
  const int VB = V / 16;
  const int NP = (VB + 1) / 2;
  const int ch = blockIdx.x;
  const int head = ch / s.Nc, ci = ch % s.Nc;
  const int b = head / s.H, h = head % s.H;
  const int t0 = ci * C;
  const size_t tok0 = seq_begin(s, b);
  s.T = seq_len(s, b);  // this sequence's length from here on
  if (t0 >= s.T) return;  // past the end of a shorter packed sequence
  const size_t krs = (size_t)s.H * KD, vrs = (size_t)s.H * V;
  const T* Kg = (const T*)in.k + (tok0 * s.H + h) * KD;
  const T* Qg = (const T*)in.q + (tok0 * s.H + h) * KD;
  const T* dOg = (const T*)dOv + (tok0 * s.H + h) * (size_t)V;
  const float* dWg = bb.dW + (size_t)ch * C * V;
  const float* Ug = sv.U + (size_t)ch * C * V;

  // Stage A-operand columns [c0, c0 + ncols) (ncols a multiple of 32) into LDS
  // columns [0, ncols); columns at or beyond V, and rows past T, are zero.
  auto stage = [&](int c0, int ncols) {
    constexpr int IT = (C * Sm::NCOL / 8 + NTHR - 1) / NTHR;
    const int n8 = ncols / 8;
    Raw8<T> ro[IT];
    f32x4 rw[IT][2], ru[IT][2];
    // unconditional loads from clamped positions (masked below), so that
    // every load of the batch is in flight before the first wait
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = min(tid + NTHR * it, C * n8 - 1);
      const int r = idx / n8, col = min(c0 + 8 * (idx % n8), V - 8);
      ro[it] = load8(dOg + (size_t)min(t0 + r, s.T - 1) * vrs + col);
      const float* pw = dWg + (size_t)r * V + col;
      const float* pu = Ug + (size_t)r * V + col;
      rw[it][0] = *(const f32x4*)pw;
      rw[it][1] = *(const f32x4*)(pw + 4);
      ru[it][0] = *(const f32x4*)pu;
      ru[it][1] = *(const f32x4*)(pu + 4);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + NTHR * it;
      if (idx >= C * n8) continue;
      const int r = idx / n8, c = 8 * (idx % n8);
      const bool cok = c0 + c < V;
      const Raw8<T> dov = (cok && t0 + r < s.T) ? ro[it] : zero_raw8<T>();
      const f32x4 w0 = cok ? rw[it][0] : zero4(), w1 = cok ? rw[it][1] : zero4();
      const f32x4 u0 = cok ? ru[it][0] : zero4(), u1 = cok ? ru[it][1] : zero4();
      if constexpr (SPLIT) {
        *(uint4*)&sm.dO[r][c] = dov.w[0];
        bf16x4 h0, l0, h1, l1;
        split_frag(w0, h0, l0);
        split_frag(w1, h1, l1);
        *(bf16x8*)&sm.dWh[r][c] = __builtin_shufflevector(h0, h1, 0, 1, 2, 3, 4, 5, 6, 7);
        *(bf16x8*)&sm.dWl[r][c] = __builtin_shufflevector(l0, l1, 0, 1, 2, 3, 4, 5, 6, 7);
        split_frag(u0, h0, l0);
        split_frag(u1, h1, l1);
        *(bf16x8*)&sm.Uh[r][c] = __builtin_shufflevector(h0, h1, 0, 1, 2, 3, 4, 5, 6, 7);
        *(bf16x8*)&sm.Ul[r][c] = __builtin_shufflevector(l0, l1, 0, 1, 2, 3, 4, 5, 6, 7);
      } else {
        lds_put_raw8(&sm.dO[r][c], dov);
        *(f32x4*)&sm.dWh[r][c] = w0;
        *(f32x4*)&sm.dWh[r][c + 4] = w1;
        *(f32x4*)&sm.Uh[r][c] = u0;
        *(f32x4*)&sm.Uh[r][c + 4] = u1;
      }
    }
  };

  // rows of Q and K at the accumulator positions (row 16 rt + 4 g + j, key
  // 16 ct + n); bf16 values are kept as packed pairs
  constexpr int QW = sizeof(T) == 2 ? 2 : 4;  // 32-bit words per 4 values
  uint32_t qv[RTW][CTW][QW], kv[RTW][CTW][QW];
#pragma unroll
  for (int i = 0; i < RTW; ++i)
#pragma unroll
    for (int c = 0; c < CTW; ++c) {
      const int ct = q * CTW + c, rt = min(rt0 + i, NT - 1);
#pragma unroll
      for (int j = 0; j < QW; ++j) qv[i][c][j] = kv[i][c][j] = 0u;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = t0 + 16 * rt + 4 * g + j;
        const bool ok = rows && ct < KT && t < s.T;
        const size_t off = (size_t)min(t, s.T - 1) * krs + key_of_row<KD>(16 * min(ct, KT - 1) + n);
        if constexpr (sizeof(T) == 2) {
          const uint32_t qx = (uint32_t)((const uint16_t*)Qg)[off] << (16 * (j & 1));
          const uint32_t kx = (uint32_t)((const uint16_t*)Kg)[off] << (16 * (j & 1));
          qv[i][c][j >> 1] |= ok ? qx : 0u;
          kv[i][c][j >> 1] |= ok ? kx : 0u;
        } else {
          const uint32_t qx = __float_as_uint(((const float*)Qg)[off]);
          const uint32_t kx = __float_as_uint(((const float*)Kg)[off]);
          qv[i][c][j] = ok ? qx : 0u;
          kv[i][c][j] = ok ? kx : 0u;
        }
      }
    }
  auto unpack = [&](const uint32_t (&x)[QW], int j) -> float {
    if constexpr (sizeof(T) == 2) return __uint_as_float((j & 1) ? (x[j >> 1] & 0xffff0000u) : (x[j >> 1] << 16));
    else return __uint_as_float(x[j]);
  };
  // coefficient vectors: loaded with the staged rows (one memory latency for
  // both), stored to LDS after the staging has waited for them
  constexpr int NCF = (3 * E * C / 4 + NTHR - 1) / NTHR;
  f32x4 cf[NCF];
  {
    const float* cg = p.coef + (size_t)ch * 3 * E * C;
#pragma unroll
    for (int i = 0; i < NCF; ++i)
      cf[i] = *(const f32x4*)(cg + 4 * min(tid + NTHR * i, 3 * E * C / 4 - 1));
  }
  if constexpr (Sm::STAGE_ALL) stage(0, 32 * NP);
#pragma unroll
  for (int i = 0; i < NCF; ++i)
    if (tid + NTHR * i < 3 * E * C / 4) *(f32x4*)(&sm.coef[0][0][0] + 4 * (tid + NTHR * i)) = cf[i];

  // B operands: S_e^T and dS'_e^T for this wave's key columns; lane (g, n)
  // takes key row 16 ct + n of value block 2 pp + g / 2, columns 8 (g & 1) + 0..7
  // (loads from clamped tiles, never under a per-lane branch: a value block
  // past V meets zero A-operand columns, and the state-gradient dot product
  // below masks it)
  const T* Sck = (const T*)sv.Sck;
  const T* dSck = (const T*)bb.dSck;
  const T* dSlk = (const T*)bb.dSck_lo;
  Raw8<T> sbuf[CTW][NPMAX], dbuf[CTW][NPMAX], dlbuf[PDS ? CTW : 1][PDS ? NPMAX : 1];
  auto load_pair = [&](int e, int c, int pp) {
    const int ct = min(q * CTW + c, KT - 1);
    const int vb = min(2 * pp + (g >> 1), VB - 1);
    const size_t off = ((((size_t)ch * E + e) * VB + vb) * KD + 16 * ct + n) * 16 + 8 * (g & 1);
    sbuf[c][pp] = load8(Sck + off);
    dbuf[c][pp] = load8(dSck + off);
    if constexpr (PDS) dlbuf[c][pp] = load8(dSlk + off);
  };
#pragma unroll
  for (int pp = 0; pp < NPMAX; ++pp)
#pragma unroll
    for (int c = 0; c < CTW; ++c)
      if (pp < NP) load_pair(0, c, pp);
  __syncthreads();

  f32x4 dq[RTW][CTW], dk[RTW][CTW];
#pragma unroll
  for (int i = 0; i < RTW; ++i)
#pragma unroll
    for (int c = 0; c < CTW; ++c) {
      dq[i][c] = zero4();
      dk[i][c] = zero4();
    }

  for (int e = 0; e < E; ++e) {
    float gpart = 0.f;
    f32x4 X[RTW][CTW], Y[RTW][CTW], Vp[RTW][CTW];
#pragma unroll
    for (int i = 0; i < RTW; ++i)
#pragma unroll
      for (int c = 0; c < CTW; ++c) {
        X[i][c] = zero4();
        Y[i][c] = zero4();
        Vp[i][c] = zero4();
      }
#pragma unroll
    for (int pp = 0; pp < NPMAX; ++pp) {
      if (pp >= NP) continue;
      int col = 32 * pp;
      if constexpr (!Sm::STAGE_ALL) {
        __syncthreads();
        stage(32 * pp, 32);
        __syncthreads();
        col = 0;
      }
      if (w < 4) {  // the state-gradient dot product, once per key quarter
#pragma unroll
        for (int c = 0; c < CTW; ++c) {
          if (q * CTW + c >= KT) continue;
          float a[8], d[8], part = 0.f;
          raw8_to_f(sbuf[c][pp], a);
          raw8_to_f(dbuf[c][pp], d);
          if constexpr (PDS) {
            float dl[8];
            raw8_to_f(dlbuf[c][pp], dl);
#pragma unroll
            for (int i = 0; i < 8; ++i) d[i] += dl[i];
          }
#pragma unroll
          for (int i = 0; i < 8; ++i) part += a[i] * d[i];
          gpart += (2 * pp + (g >> 1) < VB) ? part : 0.f;
        }
      }
      if (rows) {
#pragma unroll
        for (int i = 0; i < RTW; ++i) {
          const int r = 16 * (rt0 + i) + n;
          const int cc = col + 8 * g;
          const Raw8<T> ao = *(const Raw8<T>*)&sm.dO[r][cc];
          const Raw8<T> awh = *(const Raw8<T>*)&sm.dWh[r][cc];
          const Raw8<T> auh = *(const Raw8<T>*)&sm.Uh[r][cc];
          Raw8<T> awl, aul;
          if constexpr (SPLIT) {
            awl = *(const Raw8<T>*)&sm.dWl[r][cc];
            aul = *(const Raw8<T>*)&sm.Ul[r][cc];
          }
#pragma unroll
          for (int c = 0; c < CTW; ++c) {
            if (q * CTW + c >= KT) continue;
            mma8(X[i][c], ao, sbuf[c][pp]);
            mma8(Y[i][c], awh, sbuf[c][pp]);
            mma8(Vp[i][c], auh, dbuf[c][pp]);
            if constexpr (SPLIT) {
              mma8(Y[i][c], awl, sbuf[c][pp]);
              mma8(Vp[i][c], aul, dbuf[c][pp]);
            }
            if constexpr (PDS) mma8(Vp[i][c], auh, dlbuf[c][pp]);
          }
        }
      }
      // this pair is done for slice e: fetch it for slice e + 1
      if (e + 1 < E) {
#pragma unroll
        for (int c = 0; c < CTW; ++c) load_pair(e + 1, c, pp);
      }
    }
    // fold slice e into dq_s, dk_s; per-row sums of Q o X, K o Y, K o V'
    const int par = e & 1;
    float rs[3][16];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int j = 0; j < 4; ++j) rs[0][4 * i + j] = rs[1][4 * i + j] = rs[2][4 * i + j] = 0.f;
      if (i >= RTW || !rows) continue;
      const int rt = rt0 + i;
      const f32x4 ca = *(const f32x4*)&sm.coef[0][e][16 * rt + 4 * g];
      const f32x4 cb = *(const f32x4*)&sm.coef[1][e][16 * rt + 4 * g];
      const f32x4 cc = *(const f32x4*)&sm.coef[2][e][16 * rt + 4 * g];
#pragma unroll
      for (int c = 0; c < CTW; ++c) {
        if (q * CTW + c >= KT) continue;
        dq[i][c] += cb * X[i][c];
        dk[i][c] += ca * Y[i][c] + cc * Vp[i][c];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float kj = unpack(kv[i][c], j), qj = unpack(qv[i][c], j);
          rs[0][4 * i + j] += kj * Y[i][c][j];   // d a_e
          rs[1][4 * i + j] += qj * X[i][c][j];   // d b_e
          rs[2][4 * i + j] += kj * Vp[i][c][j];  // d c_e
        }
      }
    }
    // lane n of group g now receives the row sum of row 16 (rt0 + n / 4) + 4 g + n % 4
    const int rrow = 16 * (rt0 + (n >> 2)) + 4 * g + (n & 3);
#pragma unroll
    for (int kind = 0; kind < 3; ++kind) {
      const float x = group16_transpose_sum(rs[kind], n);
      if (rows && (n >> 2) < RTW) sm.red[par][q][kind][rrow] = x;
    }
    if (w < 4) {
      gpart = wave_sum(gpart);
      if (l == 0) sm.gred[q][e] = gpart;
    }
    __syncthreads();
    for (int idx = tid; idx < 3 * C; idx += NTHR) {  // fixed-order sum over the key quarters
      const int kind = idx / C, r = idx % C;
      sm.dcf[kind][e][r] = ((sm.red[par][0][kind][r] + sm.red[par][1][kind][r]) +
                            sm.red[par][2][kind][r]) + sm.red[par][3][kind][r];
    }
  }
  __syncthreads();
  for (int idx = tid; idx < 3 * E * C; idx += NTHR)
    bb.dcoef[(size_t)ch * 3 * E * C + idx] = (&sm.dcf[0][0][0])[idx];
  if (tid < E4)
    bb.dgC[(size_t)ch * E4 + tid] =
        (tid < E) ? ((sm.gred[0][tid] + sm.gred[1][tid]) + sm.gred[2][tid]) + sm.gred[3][tid] : 0.f;
  if (rows) {
#pragma unroll
    for (int i = 0; i < RTW; ++i)
#pragma unroll
      for (int c = 0; c < CTW; ++c) {
        const int ct = q * CTW + c, rt = rt0 + i;
        if (ct >= KT) continue;
        const int key = key_of_row<KD>(16 * ct + n);  // the key of tile row 16 ct + n
        float* qo = bb.dqs + (size_t)ch * C * KD + (size_t)(16 * rt + 4 * g) * KD + key;
        float* ko = bb.dks + (size_t)ch * C * KD + (size_t)(16 * rt + 4 * g) * KD + key;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          qo[(size_t)j * KD] = dq[i][c][j];
          ko[(size_t)j * KD] = dk[i][c][j];
        }
      }
  }
}

// ========================================================= per-chunk gradients
// fp32 x fp32 products on MFMA: bf16 operands split into hi + lo (three
// products), fp32 operands on the fp32 MFMA.
__device__ __forceinline__ void mma_ff(f32x4& acc, f32x4 a, f32x4 b, bf16_t*) {
  bf16x4 ah, al, bh, bl;
  split_frag(a, ah, al);
  split_frag(b, bh, bl);
  mma16(acc, ah, bh);
  mma16(acc, ah, bl);
  mma16(acc, al, bh);
}
__device__ __forceinline__ void mma_ff(f32x4& acc, f32x4 a, f32x4 b, float*) { mma16(acc, a, b); }
// fp32 A times an exactly representable B (an input)
__device__ __forceinline__ void mma_fx(f32x4& acc, f32x4 a, f32x4 b, bf16_t*) {
  bf16x4 ah, al;
  split_frag(a, ah, al);
  const bf16x4 bb = cvt_frag<bf16_t>(b);
  mma16(acc, ah, bb);
  mma16(acc, al, bb);
}
__device__ __forceinline__ void mma_fx(f32x4& acc, f32x4 a, f32x4 b, float*) { mma16(acc, a, b); }

// 8-value fp32 pieces as (hi, lo) bf16 pairs
__device__ __forceinline__ void split8(f32x4 x0, f32x4 x1, Raw8<bf16_t>& hi, Raw8<bf16_t>& lo) {
  bf16x4 h0, l0, h1, l1;
  split_frag(x0, h0, l0);
  split_frag(x1, h1, l1);
  hi.w[0] = __builtin_bit_cast(uint4, __builtin_shufflevector(h0, h1, 0, 1, 2, 3, 4, 5, 6, 7));
  lo.w[0] = __builtin_bit_cast(uint4, __builtin_shufflevector(l0, l1, 0, 1, 2, 3, 4, 5, 6, 7));
}
// 32-deep step: exact operand a (an input) times fp32 values b (split for bf16)
__device__ __forceinline__ void mma8_xs(f32x4& acc, const Raw8<bf16_t>& a, f32x4 b0, f32x4 b1) {
  Raw8<bf16_t> bh, bl;
  split8(b0, b1, bh, bl);
  mma8(acc, a, bh);
  mma8(acc, a, bl);
}
__device__ __forceinline__ void mma8_xs(f32x4& acc, const Raw8<float>& a, f32x4 b0, f32x4 b1) {
  mma16(acc, __builtin_bit_cast(f32x4, a.w[0]), b0);
  mma16(acc, __builtin_bit_cast(f32x4, a.w[1]), b1);
}
// 32-deep step, fp32 x fp32 (three bf16 products, or fp32 MFMAs)
__device__ __forceinline__ void mma8_ss(f32x4& acc, f32x4 a0, f32x4 a1, f32x4 b0, f32x4 b1,
                                        bf16_t*) {
  Raw8<bf16_t> ah, al, bh, bl;
  split8(a0, a1, ah, al);
  split8(b0, b1, bh, bl);
  mma8(acc, ah, bh);
  mma8(acc, ah, bl);
  mma8(acc, al, bh);
}
__device__ __forceinline__ void mma8_ss(f32x4& acc, f32x4 a0, f32x4 a1, f32x4 b0, f32x4 b1,
                                        float*) {
  mma16(acc, a0, b0);
  mma16(acc, a1, b1);
}
// fp32 A (split for bf16) times two exact 16-deep B fragments: a 32-deep step
__device__ __forceinline__ void mma_fx2(f32x4& acc, f32x4 a0, f32x4 a1, bf16x4 b0, bf16x4 b1) {
  bf16x4 h0, l0, h1, l1;
  split_frag(a0, h0, l0);
  split_frag(a1, h1, l1);
  mma32(acc, h0, h1, b0, b1);
  mma32(acc, l0, l1, b0, b1);
}
__device__ __forceinline__ void mma_fx2(f32x4& acc, f32x4 a0, f32x4 a1, f32x4 b0, f32x4 b1) {
  mma16(acc, a0, b0);
  mma16(acc, a1, b1);
}
// 8 gradient values to an out_dtype row
__device__ __forceinline__ void store8_out(void* base, size_t off, f32x4 a, f32x4 b, int out_bf16) {
  if (out_bf16) {
    const bf16x4 h0 = cvt_frag<bf16_t>(a), h1 = cvt_frag<bf16_t>(b);
    *(uint4*)((bf16_t*)base + off) =
        __builtin_bit_cast(uint4, __builtin_shufflevector(h0, h1, 0, 1, 2, 3, 4, 5, 6, 7));
  } else {
    *(f32x4*)((float*)base + off) = a;
    *(f32x4*)((float*)base + off + 4) = b;
  }
}

// 4 gradient values (consecutive columns of one row) to an out_dtype row
__device__ __forceinline__ void store4_out(void* base, size_t off, f32x4 a, int out_bf16) {
  if (out_bf16)
    *(bf16x4*)((bf16_t*)base + off) = cvt_frag<bf16_t>(a);
  else
    *(f32x4*)((float*)base + off) = a;
}

// LDS plan of the per-chunk kernel.  C x C fp32 matrices use a row stride of
// C + 4 floats (16-byte rows, conflict-free fragment reads).  Two regions are
// reused once their first contents are dead: the Q / K rows become dM^T and
// dA_kk + dA_kk^T, and R / (I + L)^{-1} become K^T / Q^T (bf16 instances;
// fp32 ones read Q and K from global memory so that the plan fits 160 KiB).
template <typename T, int KD, int C, int E>
struct ChunkSmem {
  static constexpr int CP = C + 4;
  static constexpr int KP = KD + 8;
  static constexpr int CT = C + 4;
  static constexpr int NT = C / 16;
  static constexpr bool STAGE_QK = sizeof(T) == 2;
  static constexpr int QR = STAGE_QK ? C : 1;
  static constexpr int KR = STAGE_QK ? KD : 1;
  // dT later holds three C x E sums of the Gram backward: at least C rows,
  // more where 3 C E exceeds C x CP (wide second keys at small chunks)
  static constexpr int DT_ROWS = 3 * C * E > C * CP ? (3 * C * E + CP - 1) / CP : C;
  union U1 {
    struct { T sQ[QR][KP]; T sK[QR][KP]; } qk;           // Q, K rows
    struct { float dMT[C][CP]; float Dsym[C][CP]; } tr;  // dA_qk^T, dA_kk + dA_kk^T
  };
  union U2 {
    struct { float R[C][CP]; float X1[C][CP]; } r;       // R; (I + L)^{-1}, then dL o A_hat
    struct { T Kt[KR][CT]; T Qt[KR][CT]; } kq;           // K^T, Q^T
  };
  alignas(16) U1 u1;
  alignas(16) U2 u2;
  alignas(16) float Aqk[C][CP];  // A_qk, then dR' = dM o A_qk
  alignas(16) float Akk[C][CP];  // A_kk, then dR = dA_hat o A_kk
  alignas(16) float dM[C][CP];   // dA_qk = dM o R'
  alignas(16) float dT[DT_ROWS][CP];  // dTu, P = N^{-T} dTu, dA_kk; then the Gram-backward sums
  alignas(16) float Y[NT > 1 ? NT - 1 : 1][16][17];
  alignas(16) float q2[C][E];
  alignas(16) float k2[C][E];
  alignas(16) double G[C][E];
  alignas(16) float dG[C][E];
  alignas(16) float beta[C];
  alignas(16) float dbeta[C];
};

// Eight waves (two per SIMD): every phase is latency-bound at this size, so
// the second wave per SIMD hides LDS and memory latency of the first.
constexpr int CHUNK_NW = 8;
constexpr int CHUNK_NTHR = CHUNK_NW * 64;

template <typename T, int KD, int C, int E>
__global__ __launch_bounds__(CHUNK_NTHR) void k_bwd_chunk(Shape s, FwdIn in, const void* dOv,
                                                   PrepBufs p, SavedBufs sv, BwdBufs bb, void* dqv, void* dkv,
                                                   void* dvv, void* dq2v, void* dk2v, float* dg,
                                                   float* dbeta) {
  constexpr int NT = C / 16;
  constexpr int KT = KD / 16;
  constexpr int E4 = (E + 3) & ~3;
  constexpr int NVPMAX = 4;  // pairs of 16-column value blocks, V <= 128
  constexpr int NW = CHUNK_NW, NTHR = CHUNK_NTHR;
  typedef typename Elem<T>::frag F;
  typedef ChunkSmem<T, KD, C, E> Sm;
  constexpr bool STAGE_QK = Sm::STAGE_QK;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Sm& sm = *reinterpret_cast<Sm*>(smem_raw);
  T* tag = nullptr;  // selects the MFMA flavour of the mixed-precision helpers
  const int tid = threadIdx.x, w = wave_id(), l = lane_id(), g = l >> 4, n = l & 15;
  const int V = s.V;
  const int NVP = (V / 16 + 1) / 2;
  const int ch = blockIdx.x;
  const int head = ch / s.Nc, ci = ch % s.Nc;
  const int b = head / s.H, h = head % s.H;
  const int t0 = ci * C;
  const size_t tok0 = seq_begin(s, b);
  s.T = seq_len(s, b);  // this sequence's length from here on
  if (t0 >= s.T) return;  // past the end of a shorter packed sequence
  const size_t krs = (size_t)s.H * KD, vrs = (size_t)s.H * V;
  const T* Kg = (const T*)in.k + (tok0 * s.H + h) * KD;
  const T* Qg = (const T*)in.q + (tok0 * s.H + h) * KD;
  const T* Vg = (const T*)in.v + (tok0 * s.H + h) * (size_t)V;
  const T* dOg = (const T*)dOv + (tok0 * s.H + h) * (size_t)V;
  const float* Ug = sv.U + (size_t)ch * C * V;
  const float* Xg = sv.X + (size_t)ch * C * V;
  const float* dUg = bb.dU + (size_t)ch * C * V;
  const float* dWg = bb.dW + (size_t)ch * C * V;
  const float* dcf = bb.dcoef + (size_t)ch * 3 * E * C;
  const size_t eoff = (tok0 * s.H + h) * E;
  const size_t erow = (size_t)s.H * E;
  const bool gdn = s.variant == 1;

  // ---- phase 0: per-position vectors, Q and K rows, in-chunk cumulative
  // log-gates.  Every global load of the phase is issued before the first of
  // their results is stored (one memory latency instead of one per array),
  // and so are the loads of dv, which needs nothing the kernel computes.
  constexpr int NQE = (C * E + NTHR - 1) / NTHR;             // q2, k2 entries per thread
  constexpr int IT = STAGE_QK ? (C * KD / 8 + NTHR - 1) / NTHR : 1;  // Q, K pieces
  constexpr int NNV = (C * C / 4 + NTHR - 1) / NTHR;        // (I + L)^{-1} pieces
  constexpr int NGE = (E + NW - 1) / NW;                     // slices per wave (g)
  constexpr int IDV = (C * 128 / 8 + NTHR - 1) / NTHR;      // 8-value pieces of dv
  const bool have_ninv = gdn && p.ninv != nullptr;
  float q2v[NQE], k2v[NQE], bv = 0.f;
  Raw8<T> qv[IT], kv[IT];
  f32x4 nv[NNV];
  double gv[NGE];
  f32x4 dvx[IDV][2];
#pragma unroll
  for (int i = 0; i < NQE; ++i) {
    const int idx = tid + NTHR * i, r = idx / E, e = idx % E, t = t0 + r;
    const bool ok = idx < C * E && t < s.T;
    q2v[i] = ok ? ld_f((const T*)in.q2 + eoff + (size_t)t * erow + e) : 0.f;
    k2v[i] = ok ? ld_f((const T*)in.k2 + eoff + (size_t)t * erow + e) : 0.f;
  }
  if (tid < C) {
    const int t = t0 + tid;
    bv = (t < s.T) ? (in.beta ? in.beta[(tok0 + t) * s.H + h] : 1.f) : 0.f;
  }
  if constexpr (STAGE_QK) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + NTHR * it;
      const int r = idx / (KD / 8), c8 = idx % (KD / 8);
      const int t = t0 + r;
      qv[it] = zero_raw8<T>();
      kv[it] = zero_raw8<T>();
      if (idx < C * KD / 8 && t < s.T) {
        qv[it] = load8(Qg + (size_t)t * krs + 8 * c8);
        kv[it] = load8(Kg + (size_t)t * krs + 8 * c8);
      }
    }
  }
  // (I + L)^{-1} as the forward's prep kernel formed it (GDN): into its LDS
  // region, which stays free until the solve backward
  if (have_ninv) {
    const float* src = p.ninv + (size_t)ch * C * C;
#pragma unroll
    for (int i = 0; i < NNV; ++i) {
      const int idx = tid + NTHR * i;
      nv[i] = idx < C * C / 4 ? *(const f32x4*)(src + 4 * idx) : zero4();
    }
  }
#pragma unroll
  for (int i = 0; i < NGE; ++i) {
    const int e = w + NW * i, t = t0 + l;
    gv[i] = (e < E && l < C && t < s.T) ? (double)in.g[eoff + (size_t)t * erow + e] : 0.0;
  }
  // rows of dv = Tu^T dU = -dW (GDN) or diag(beta) dU (sGLA), 8 values a piece
#pragma unroll
  for (int it = 0; it < IDV; ++it) {
    const int idx = tid + NTHR * it, n8 = V / 8;
    const int r = idx / n8, c = 8 * (idx % n8);
    dvx[it][0] = dvx[it][1] = zero4();
    if (idx < C * n8 && t0 + r < s.T) {
      const float* src = (gdn ? dWg : dUg) + (size_t)r * V + c;
      dvx[it][0] = *(const f32x4*)src;
      dvx[it][1] = *(const f32x4*)(src + 4);
    }
  }
  // ---- the stores
#pragma unroll
  for (int i = 0; i < NQE; ++i) {
    const int idx = tid + NTHR * i;
    if (idx < C * E) {
      sm.q2[idx / E][idx % E] = q2v[i];
      sm.k2[idx / E][idx % E] = k2v[i];
    }
  }
  if (tid < C) sm.beta[tid] = bv;
  if constexpr (STAGE_QK) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + NTHR * it;
      if (idx >= C * KD / 8) continue;
      const int r = idx / (KD / 8), c8 = idx % (KD / 8);
      *(Raw8<T>*)&sm.u1.qk.sQ[r][8 * c8] = qv[it];
      *(Raw8<T>*)&sm.u1.qk.sK[r][8 * c8] = kv[it];
    }
  }
  if (have_ninv) {
#pragma unroll
    for (int i = 0; i < NNV; ++i) {
      const int idx = tid + NTHR * i;
      if (idx < C * C / 4) *(f32x4*)&sm.u2.r.X1[idx / (C / 4)][4 * (idx % (C / 4))] = nv[i];
    }
  }
  // G = inclusive cumulative sum of g over the chunk, in fp64: one wave per
  // slice, lane r holds row r
#pragma unroll
  for (int i = 0; i < NGE; ++i) {
    const int e = w + NW * i;
    if (e >= E) continue;  // wave-uniform
    double x = gv[i];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double y = __shfl_up(x, off, 64);
      if (l >= off) x += y;
    }
    if (l < C) sm.G[l][e] = x;
  }
  __syncthreads();

  // ---- dv = Tu^T dU = -dW (GDN) or diag(beta) dU (sGLA)
#pragma unroll
  for (int it = 0; it < IDV; ++it) {
    const int idx = tid + NTHR * it, n8 = V / 8;
    const int r = idx / n8, c = 8 * (idx % n8);
    const int t = t0 + r;
    if (idx >= C * n8 || t >= s.T) continue;
    const float sc = gdn ? -1.f : sm.beta[r];
    store8_out(dvv, ((tok0 + t) * s.H + h) * (size_t)V + c, sc * dvx[it][0], sc * dvx[it][1],
               s.out_bf16);
  }

  // Q / K rows as 8-element operands at columns [col, col + 8) (zero past KD or T)
  auto qrow8 = [&](int r, int col) -> Raw8<T> {
    if (col >= KD) return zero_raw8<T>();
    if constexpr (STAGE_QK) return *(const Raw8<T>*)&sm.u1.qk.sQ[r][col];
    else return (t0 + r < s.T) ? load8(Qg + (size_t)(t0 + r) * krs + col) : zero_raw8<T>();
  };
  auto krow8 = [&](int r, int col) -> Raw8<T> {
    if (col >= KD) return zero_raw8<T>();
    if constexpr (STAGE_QK) return *(const Raw8<T>*)&sm.u1.qk.sK[r][col];
    else return (t0 + r < s.T) ? load8(Kg + (size_t)(t0 + r) * krs + col) : zero_raw8<T>();
  };

  // ---- phase 1, per 16 x 16 tile (rt, st); lane (g, n) holds rows 16 rt + 4 g + j
  // of column 16 st + n:  A_qk, A_kk, dM = dO U^T (lower), dTu = dU X^T (GDN),
  // then R', R and  dR' = dM o A_qk, dA_qk = dM o R'  element by element
  // tiles in the order: the NT (NT + 1) / 2 lower ones, then the upper ones,
  // dealt round-robin to the waves
  for (int tile = w; tile < NT * NT; tile += NW) {
    constexpr int NL = NT * (NT + 1) / 2;
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
    const bool lower = st <= rt;
    const int ra = 16 * rt + n, cb = 16 * st + n;  // A-operand row, B-operand row
    const bool raok = t0 + ra < s.T;
    // global operand loads first (value columns 32 vp + 8 g .. + 7)
    Raw8<T> dOa[NVPMAX];
    f32x4 Ub[NVPMAX][2], dUa[NVPMAX][2], Xb[NVPMAX][2];
    // (unconditional loads from clamped positions under wave-uniform
    // conditions only, masked once the values are used)
#pragma unroll
    for (int vp = 0; vp < NVPMAX; ++vp) {
      const int col = min(32 * vp + 8 * g, V - 8);
      dOa[vp] = zero_raw8<T>();
      Ub[vp][0] = Ub[vp][1] = dUa[vp][0] = dUa[vp][1] = Xb[vp][0] = Xb[vp][1] = zero4();
      if (vp >= NVP) continue;
      if (lower) {
        dOa[vp] = load8(dOg + (size_t)min(t0 + ra, s.T - 1) * vrs + col);
        Ub[vp][0] = *(const f32x4*)(Ug + (size_t)cb * V + col);
        Ub[vp][1] = *(const f32x4*)(Ug + (size_t)cb * V + col + 4);
      }
      if (gdn && lower) {
        dUa[vp][0] = *(const f32x4*)(dUg + (size_t)ra * V + col);
        dUa[vp][1] = *(const f32x4*)(dUg + (size_t)ra * V + col + 4);
        Xb[vp][0] = *(const f32x4*)(Xg + (size_t)cb * V + col);
        Xb[vp][1] = *(const f32x4*)(Xg + (size_t)cb * V + col + 4);
      }
    }
    f32x4 aq = zero4(), ak = zero4(), dm = zero4(), dt = zero4();
    if (lower) {
#pragma unroll
      for (int kp = 0; kp < (KD + 31) / 32; ++kp) {
        const int col = 32 * kp + 8 * g;
        const Raw8<T> kb = krow8(cb, col);
        mma8(aq, qrow8(ra, col), kb);
        mma8(ak, krow8(ra, col), kb);
      }
    }
    // decayed Grams of the lane's four (r, c) pairs (formed for every pair of
    // a lower tile and masked afterwards: no per-lane branch around the
    // shared-memory reads, which are whole-row vector reads)
    float rq[4] = {0.f, 0.f, 0.f, 0.f}, rk[4] = {0.f, 0.f, 0.f, 0.f};
    if (lower) {
      const int c = 16 * st + n;
      double Gc[E];
      float k2c[E];
      lds_row<E>(Gc, &sm.G[c][0]);
      lds_row<E>(k2c, &sm.k2[c][0]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 16 * rt + 4 * g + j;
        double Gr[E];
        float q2r[E], k2r[E];
        lds_row<E>(Gr, &sm.G[r][0]);
        lds_row<E>(q2r, &sm.q2[r][0]);
        lds_row<E>(k2r, &sm.k2[r][0]);
        float aq = 0.f, ak = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float d = exp_nonpos((float)(Gr[e] - Gc[e])) * k2c[e];
          aq += q2r[e] * d;
          ak += k2r[e] * d;
        }
        rq[j] = (c <= r) ? aq : 0.f;
        rk[j] = (c <= r) ? ak : 0.f;
      }
    }
    if (lower) {
#pragma unroll
      for (int vp = 0; vp < NVPMAX; ++vp) {
        if (vp >= NVP) continue;
        const bool cok = 32 * vp + 8 * g < V;  // columns past V (odd V / 16) contribute zero
        mma8_xs(dm, (cok && raok) ? dOa[vp] : zero_raw8<T>(), Ub[vp][0], Ub[vp][1]);
      }
    }
    // dTu only on and below the diagonal: Tu is lower triangular, and of
    // P = N^{-T} dTu the solve below uses the diagonal (dbeta) and the
    // strictly lower part (dL), which read only those tiles of dTu
    if (gdn && lower) {
#pragma unroll
      for (int vp = 0; vp < NVPMAX; ++vp) {
        if (vp >= NVP) continue;
        const bool cok = 32 * vp + 8 * g < V;
        mma8_ss(dt, cok ? dUa[vp][0] : zero4(), cok ? dUa[vp][1] : zero4(), Xb[vp][0], Xb[vp][1],
                tag);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = 16 * rt + 4 * g + j, c = 16 * st + n;
      const bool le = lower && c <= r;
      sm.Aqk[r][c] = le ? dm[j] * aq[j] : 0.f;  // dR'
      sm.dM[r][c] = le ? dm[j] * rq[j] : 0.f;   // dA_qk
      sm.u2.r.R[r][c] = (lower && c < r) ? rk[j] : 0.f;
      sm.Akk[r][c] = ak[j];
      sm.dT[r][c] = dt[j];
    }
  }
  __syncthreads();

  if (gdn) {
    // ---- (I + L)^{-1} with L = diag(beta)(A_kk o R), strictly lower: the
    // forward's, staged in phase 0 (formed here only without it)
    if (!have_ninv)
      unit_lower_inverse<C, NTHR>(
          [&](int r, int c) { return sm.beta[r] * sm.Akk[r][c] * sm.u2.r.R[r][c]; },
          &sm.u2.r.X1[0][0], Sm::CP, &sm.Y[0][0][0]);
    // ---- P = N^{-T} dTu on MFMA (fp32 operands); N^{-T} is upper triangular.
    // Only the tiles on and below the diagonal are formed: dbeta takes the
    // diagonal and dL the strictly lower part (the others would stay unused)
    f32x4 pt[(NT * NT + NW - 1) / NW];
#pragma unroll
    for (int i = 0; i < (NT * NT + NW - 1) / NW; ++i) {
      const int tile = w + NW * i;
      f32x4 acc = zero4();
      if (tile < NT * NT && tile % NT <= tile / NT) {
        const int rt = tile / NT, ct = tile % NT;
        for (int kb = rt; kb < NT; ++kb) {
          f32x4 a, bv;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            a[j] = sm.u2.r.X1[16 * kb + 4 * g + j][16 * rt + n];  // (N^{-1})^T[r][k]
            bv[j] = sm.dT[16 * kb + 4 * g + j][16 * ct + n];
          }
          mma_ff(acc, a, bv, tag);
        }
      }
      pt[i] = acc;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < (NT * NT + NW - 1) / NW; ++i) {
      const int tile = w + NW * i;
      if (tile < NT * NT) {
        const int rt = tile / NT, ct = tile % NT;
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.dT[16 * rt + 4 * g + j][16 * ct + n] = pt[i][j];
      }
    }
    __syncthreads();
    if (tid < C) sm.dbeta[tid] = sm.dT[tid][tid];  // diag(N^{-T} dTu)
    // ---- dL = tril(-P Tu^T, -1) with Tu = N^{-1} diag(beta)
#pragma unroll
    for (int i = 0; i < (NT * NT + NW - 1) / NW; ++i) {
      const int tile = w + NW * i;
      f32x4 acc = zero4();
      if (tile < NT * NT) {
        const int rt = tile / NT, st = tile % NT;
        if (st <= rt) {
          for (int kb = 0; kb <= st; ++kb) {
            const f32x4 a = *(const f32x4*)&sm.dT[16 * rt + n][16 * kb + 4 * g];
            const f32x4 bv = *(const f32x4*)&sm.u2.r.X1[16 * st + n][16 * kb + 4 * g] *
                             *(const f32x4*)&sm.beta[16 * kb + 4 * g];
            mma_ff(acc, a, bv, tag);
          }
        }
      }
      pt[i] = -acc;
    }
    __syncthreads();
    // element (4g+j, n) of tile (rt, st) is dL[16 rt + 4 g + j][16 st + n]
#pragma unroll
    for (int i = 0; i < (NT * NT + NW - 1) / NW; ++i) {
      const int tile = w + NW * i;
      if (tile < NT * NT) {
        const int rt = tile / NT, st = tile % NT;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = 16 * rt + 4 * g + j, c = 16 * st + n;
          const float dl = (c < r) ? pt[i][j] : 0.f;
          const float akk = sm.Akk[r][c], rr = sm.u2.r.R[r][c];
          const float dah = sm.beta[r] * dl;
          sm.Akk[r][c] = dah * akk;          // dR
          sm.dT[r][c] = dah * rr;            // dA_kk
          sm.u2.r.X1[r][c] = dl * akk * rr;  // dL o A_hat
        }
      }
    }
    __syncthreads();
    if (tid < C) {
      float acc = 0.f;
      for (int c = 0; c < tid; ++c) acc += sm.u2.r.X1[tid][c];
      sm.dbeta[tid] += acc;
    }
  } else {
    for (int idx = tid; idx < C * C; idx += NTHR) {
      sm.Akk[idx / C][idx % C] = 0.f;  // dR
      sm.dT[idx / C][idx % C] = 0.f;   // dA_kk
    }
    // sGLA: dbeta_r = <dU_r, v_r>; four lanes per row
    if (tid < 4 * C) {
      const int r = tid >> 2, q = tid & 3, t = t0 + r;
      float acc = 0.f;
      if (t < s.T) {
        for (int c = 8 * q; c < V; c += 32) {
          const f32x4 u0 = *(const f32x4*)(dUg + (size_t)r * V + c);
          const f32x4 u1 = *(const f32x4*)(dUg + (size_t)r * V + c + 4);
          float vv[8];
          raw8_to_f(load8(Vg + (size_t)t * vrs + c), vv);
#pragma unroll
          for (int i = 0; i < 4; ++i) acc += u0[i] * vv[i] + u1[i] * vv[4 + i];
        }
      }
      acc += dpp_f<0xB1>(acc);
      acc += dpp_f<0x4E>(acc);
      if (q == 0) sm.dbeta[r] = acc;
    }
  }
  __syncthreads();

  // ---- operand layouts for dq, dk: K^T and Q^T (bf16, over the dead R / X1),
  // then dA_qk^T and dA_kk + dA_kk^T (over the dead Q / K rows)
  if constexpr (STAGE_QK) {
    constexpr int NB = (C / 4) * (KD / 4);
    for (int idx = tid; idx < 2 * NB; idx += NTHR) {
      const int m = idx / NB, bi = idx % NB;
      const int rb = bi / (KD / 4), kb = bi % (KD / 4);
      const T* src = m ? &sm.u1.qk.sQ[0][0] : &sm.u1.qk.sK[0][0];
      T* dst = m ? &sm.u2.kq.Qt[0][0] : &sm.u2.kq.Kt[0][0];
      uint2 v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = *(const uint2*)(src + (4 * rb + i) * Sm::KP + 4 * kb);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int sh = (jj & 1) * 16, wsel = jj >> 1;
        uint32_t e4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) e4[i] = ((wsel ? v[i].y : v[i].x) >> sh) & 0xffffu;
        *(uint2*)(dst + (4 * kb + jj) * Sm::CT + 4 * rb) =
            make_uint2(e4[0] | (e4[1] << 16), e4[2] | (e4[3] << 16));
      }
    }
    __syncthreads();
  }
  {
    constexpr int NB = (C / 4) * (C / 4);
    for (int idx = tid; idx < NB; idx += NTHR) {
      const int rb = idx / (C / 4), cb4 = idx % (C / 4);
      f32x4 a[4], p[4], q[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = *(const f32x4*)&sm.dM[4 * rb + i][4 * cb4];
        p[i] = *(const f32x4*)&sm.dT[4 * rb + i][4 * cb4];
        q[i] = *(const f32x4*)&sm.dT[4 * cb4 + i][4 * rb];
      }
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        f32x4 at, ds;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          at[i] = a[i][jj];
          ds[i] = p[jj][i] + q[i][jj];
        }
        *(f32x4*)&sm.u1.tr.dMT[4 * cb4 + jj][4 * rb] = at;
        *(f32x4*)&sm.u1.tr.Dsym[4 * rb + jj][4 * cb4] = ds;
      }
    }
  }
  __syncthreads();

  // K^T / Q^T fragments: rows 16 kt + n, token columns [16 sb + 4 g, + 4)
  auto ktf = [&](int kt, int sb) -> F {
    if constexpr (STAGE_QK) return ld_frag(&sm.u2.kq.Kt[16 * kt + n][16 * sb + 4 * g]);
    else {
      f32x4 x;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 16 * sb + 4 * g + j;
        x[j] = (t0 + r < s.T) ? ld_f(Kg + (size_t)(t0 + r) * krs + 16 * kt + n) : 0.f;
      }
      return cvt_frag<T>(x);
    }
  };
  auto qtf = [&](int kt, int sb) -> F {
    if constexpr (STAGE_QK) return ld_frag(&sm.u2.kq.Qt[16 * kt + n][16 * sb + 4 * g]);
    else {
      f32x4 x;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 16 * sb + 4 * g + j;
        x[j] = (t0 + r < s.T) ? ld_f(Qg + (size_t)(t0 + r) * krs + 16 * kt + n) : 0.f;
      }
      return cvt_frag<T>(x);
    }
  };

  // ---- dq = dq_s + dA_qk K;  dk = dk_s + dA_qk^T Q + (dA_kk + dA_kk^T) K
  // (the state-contraction partials dq_s, dk_s of all the wave's tiles are
  // loaded first: one memory latency instead of one per tile)
  constexpr int TPW = (NT * KT + NW - 1) / NW;  // tiles per wave
  float pqa[TPW][4], pka[TPW][4];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    const int tile = min(w + NW * i, NT * KT - 1);
    const int rt = tile % NT, kt = tile / NT;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const size_t wo = (size_t)ch * C * KD + (size_t)(16 * rt + 4 * g + j) * KD + 16 * kt + n;
      pqa[i][j] = bb.dqs[wo];
      pka[i][j] = bb.dks[wo];
    }
  }
  // bf16 operands with an even number of row tiles: every tile of the wave
  // has row tile w % NT, so the (hi, lo) splits of its dM, dA_qk^T and
  // dA_kk + dA_kk^T rows are formed once, and the results leave as one
  // quad-transposed store per lane (row 16 rt + 4 g + n % 4, four columns)
  constexpr bool HOIST = sizeof(T) == 2 && NT % 2 == 0 && NW % NT == 0;
  if constexpr (HOIST) {
    const int rt = w % NT, r = 16 * rt + n;
    bf16x4 mh[NT], ml[NT], th[NT], tl[NT], yh[NT], yl[NT];
#pragma unroll
    for (int sb = 0; sb < NT; ++sb) {
      const int c = 16 * sb + 4 * g;
      split_frag(*(const f32x4*)&sm.dM[r][c], mh[sb], ml[sb]);
      split_frag(*(const f32x4*)&sm.u1.tr.dMT[r][c], th[sb], tl[sb]);
      split_frag(*(const f32x4*)&sm.u1.tr.Dsym[r][c], yh[sb], yl[sb]);
    }
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      const int tile = w + NW * i;
      if (tile >= NT * KT) continue;  // wave-uniform
      const int kt = tile / NT;
      f32x4 aq = zero4(), ak = zero4();
#pragma unroll
      for (int sb = 0; sb < NT; sb += 2) {
        const F bk0 = ktf(kt, sb), bk1 = ktf(kt, sb + 1);
        const F bq0 = qtf(kt, sb), bq1 = qtf(kt, sb + 1);
        mma32(aq, mh[sb], mh[sb + 1], bk0, bk1);
        mma32(aq, ml[sb], ml[sb + 1], bk0, bk1);
        mma32(ak, th[sb], th[sb + 1], bq0, bq1);
        mma32(ak, tl[sb], tl[sb + 1], bq0, bq1);
        mma32(ak, yh[sb], yh[sb + 1], bk0, bk1);
        mma32(ak, yl[sb], yl[sb + 1], bk0, bk1);
      }
      f32x4 pq, pk;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        pq[j] = pqa[i][j];
        pk[j] = pka[i][j];
      }
      const f32x4 yq = quad_transpose(aq + pq, n), yk = quad_transpose(ak + pk, n);
      const int t = t0 + 16 * rt + 4 * g + (n & 3);
      if (t < s.T) {
        const size_t o = ((tok0 + t) * s.H + h) * KD + 16 * kt + 4 * (n >> 2);
        store4_out(dqv, o, yq, s.out_bf16);
        store4_out(dkv, o, yk, s.out_bf16);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    if constexpr (HOIST) break;
    const int tile = w + NW * i;
    if (tile >= NT * KT) continue;  // wave-uniform
    const int rt = tile % NT, kt = tile / NT;
    const float* pq = pqa[i];
    const float* pk = pka[i];
    f32x4 aq = zero4(), ak = zero4();
    const int r = 16 * rt + n;
#pragma unroll
    for (int sb = 0; sb + 1 < NT; sb += 2) {
      const int c0 = 16 * sb + 4 * g, c1 = c0 + 16;
      const F bk0 = ktf(kt, sb), bk1 = ktf(kt, sb + 1);
      const F bq0 = qtf(kt, sb), bq1 = qtf(kt, sb + 1);
      mma_fx2(aq, *(const f32x4*)&sm.dM[r][c0], *(const f32x4*)&sm.dM[r][c1], bk0, bk1);
      mma_fx2(ak, *(const f32x4*)&sm.u1.tr.dMT[r][c0], *(const f32x4*)&sm.u1.tr.dMT[r][c1], bq0,
              bq1);
      mma_fx2(ak, *(const f32x4*)&sm.u1.tr.Dsym[r][c0], *(const f32x4*)&sm.u1.tr.Dsym[r][c1], bk0,
              bk1);
    }
    if constexpr (NT & 1) {
      const int sb = NT - 1, c0 = 16 * sb + 4 * g;
      const F bk0 = ktf(kt, sb), bq0 = qtf(kt, sb);
      mma_fx(aq, *(const f32x4*)&sm.dM[r][c0], frag_to_f(bk0), tag);
      mma_fx(ak, *(const f32x4*)&sm.u1.tr.dMT[r][c0], frag_to_f(bq0), tag);
      mma_fx(ak, *(const f32x4*)&sm.u1.tr.Dsym[r][c0], frag_to_f(bk0), tag);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = t0 + 16 * rt + 4 * g + j;
      if (t < s.T) {
        const size_t o = ((tok0 + t) * s.H + h) * KD + 16 * kt + n;
        store_out(dqv, o, aq[j] + pq[j], s.out_bf16);
        store_out(dkv, o, ak[j] + pk[j], s.out_bf16);
      }
    }
  }

  // ---- backward of the decayed Grams R, R'.  Per slice e (one wave), lane
  // tiles of (r, c) pairs, c <= r:  d = Gamma_e[r, c] = exp(G_r[e] - G_c[e]),
  //   aq2[r] = sum_c dR'[r,c] d k2_c,   ak2[r] = sum_c dR[r,c] d k2_c,
  //   acol[c] = sum_r (dR'[r,c] q2_r + dR[r,c] k2_r) d
  static_assert(3 * C * E <= Sm::DT_ROWS * Sm::CP, "room for the three sums");
  float* aq2s = &sm.dT[0][0];  // dA_kk is dead: its space holds the three sums
  float* ak2s = aq2s + C * E;
  float* acols = ak2s + C * E;
  // the last phase's global operands go out now, under this one: the
  // coefficient-vector gradients of (r, e) = (idx / E, idx % E) and dgamma^C
  // of the wave's slices (used by lane C - 1)
  float dcfv[NQE][3], dgcv[NGE];
#pragma unroll
  for (int i = 0; i < NQE; ++i) {
    const int idx = tid + NTHR * i, r = idx / E, e = idx % E;
#pragma unroll
    for (int kind = 0; kind < 3; ++kind)
      dcfv[i][kind] = idx < C * E ? dcf[(kind * E + e) * C + r] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < NGE; ++i) {
    const int e = w + NW * i;
    dgcv[i] = (e < E && l == C - 1) ? bb.dgC[(size_t)ch * E4 + e] : 0.f;
  }
  __syncthreads();
  for (int e = w; e < E; e += NW) {
    float rowq[16], rowk[16], colacc[NT];
#pragma unroll
    for (int i = 0; i < 16; ++i) rowq[i] = rowk[i] = 0.f;
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) colacc[ct] = 0.f;
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) {
      // every shared-memory read of this row tile first (no per-lane
      // branch), then the arithmetic; pairs above the diagonal are masked by
      // selects (their exponent is positive)
      double Gr[4], Gc[NT];
      float q2r[4], k2r[4], k2c[NT], aqv[NT][4], akv[NT][4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 16 * rt + 4 * g + j;
        Gr[j] = sm.G[r][e];
        q2r[j] = sm.q2[r][e];
        k2r[j] = sm.k2[r][e];
      }
#pragma unroll
      for (int ct = 0; ct <= rt; ++ct) {
        const int c = 16 * ct + n;
        Gc[ct] = sm.G[c][e];
        k2c[ct] = sm.k2[c][e];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = 16 * rt + 4 * g + j;
          aqv[ct][j] = sm.Aqk[r][c];
          akv[ct][j] = sm.Akk[r][c];
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ct = 0; ct <= rt; ++ct) {
        const int c = 16 * ct + n;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = 16 * rt + 4 * g + j;
          const float ex = exp_nonpos((float)(Gr[j] - Gc[ct]));
          const float d = (c <= r) ? ex : 0.f;
          const float drq = aqv[ct][j] * d;
          const float drk = (c < r) ? akv[ct][j] * d : 0.f;
          rowq[4 * rt + j] += drq * k2c[ct];
          rowk[4 * rt + j] += drk * k2c[ct];
          colacc[ct] += drq * q2r[j] + drk * k2r[j];
        }
      }
    }
    // rows: sum over the 16 lanes of a group; lane n receives row 16 (n / 4) + 4 g + n % 4
    const float sq = group16_transpose_sum(rowq, n);
    const float sk = group16_transpose_sum(rowk, n);
    const int row = 16 * (n >> 2) + 4 * g + (n & 3);
    if ((n >> 2) < NT) {
      aq2s[row * E + e] = sq;
      ak2s[row * E + e] = sk;
    }
    // columns: sum over the four groups
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      float x = colacc[ct];
      x += __shfl_xor(x, 16, 64);
      x += __shfl_xor(x, 32, 64);
      if (g == 0) acols[(16 * ct + n) * E + e] = x;
    }
  }
  __syncthreads();

  // ---- per (r, e): Gram terms and the coefficient vectors
  //   a = k2 gamma, b = q2 gamma, c = k2 gamma^C / gamma
#pragma unroll
  for (int i = 0; i < NQE; ++i) {
    const int idx = tid + NTHR * i;
    if (idx >= C * E) continue;
    const int r = idx / E, e = idx % E;
    const float aq2 = aq2s[idx], ak2 = ak2s[idx], acol = acols[idx];
    const float q2 = sm.q2[r][e], k2 = sm.k2[r][e];
    const float da = dcfv[i][0], db = dcfv[i][1], dc = dcfv[i][2];
    const double G = sm.G[r][e], GC = sm.G[C - 1][e];
    const float gm = exp_nonpos((float)G), gt = exp_nonpos((float)(GC - G));
    sm.dG[r][e] = (q2 * aq2 + k2 * ak2) - acol * k2 + da * k2 * gm + db * q2 * gm - dc * k2 * gt;
    acols[idx] = dc * k2 * gt;  // this row's share of dG at the chunk end
    const int t = t0 + r;
    if (t < s.T) {
      const size_t o = eoff + (size_t)t * erow + e;
      store_out(dq2v, o, aq2 + db * gm, s.out_bf16);
      store_out(dk2v, o, ak2 + acol + da * gm + dc * gt, s.out_bf16);
    }
  }
  __syncthreads();
  // dG at the chunk end gains sum_r dc c + gamma^C dgamma^C; then dg_j = sum_{r >= j} dG_r
  // (one wave per slice, lane r holds row r)
#pragma unroll
  for (int i = 0; i < NGE; ++i) {
    const int e = w + NW * i;
    if (e >= E) continue;  // wave-uniform
    const float tail = wave_sum(l < C ? acols[l * E + e] : 0.f);
    float x = (l < C) ? sm.dG[l][e] : 0.f;
    if (l == C - 1) x += tail + exp_nonpos((float)sm.G[C - 1][e]) * dgcv[i];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_down(x, off, 64);
      if (l + off < 64) x += y;
    }
    const int t = t0 + l;
    if (l < C && t < s.T) dg[eoff + (size_t)t * erow + e] = x;
  }
  if (dbeta && tid < C) {
    const int t = t0 + tid;
    if (t < s.T) dbeta[(tok0 + t) * s.H + h] = sm.dbeta[tid];
  }
}


// ----------------------------------------------------------------- launchers
template <typename T, int KD, int C, int E>
static hipError_t rec_inst(const Shape& s, const FwdIn& in, const void* dO, const float* dSf,
                           const PrepBufs& p, const BwdBufs& bb, float* ds0, hipStream_t st) {
  constexpr int NW = bwd_waves<E>();
  const size_t smem = sizeof(RecSmem<T, KD, C, E, NW>);
  auto go = [&](auto pds_c) {
    constexpr bool PDS = decltype(pds_c)::value;
    static bool attr = false;
    if (!attr) {
      (void)hipFuncSetAttribute((const void*)k_bwd_rec<T, KD, C, E, NW, PDS>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
      attr = true;
    }
    hipLaunchKernelGGL((k_bwd_rec<T, KD, C, E, NW, PDS>), dim3(s.NH * (s.V / 16)), dim3(NW * 64),
                       smem, st, s, in, dO, dSf, p, bb, ds0);
    return hipGetLastError();
  };
  if (sizeof(T) == 2 && bb.dSck_lo) return go(std::integral_constant<bool, sizeof(T) == 2>{});
  return go(std::integral_constant<bool, false>{});
}

template <typename T, int KD, int C, int E>
static hipError_t state_inst(const Shape& s, const FwdIn& in, const void* dO, const PrepBufs& p,
                             const SavedBufs& sv, const BwdBufs& bb, hipStream_t st) {
  const size_t smem = sizeof(StateSmem<T, KD, C, E>);
  auto go = [&](auto pds_c) {
    constexpr bool PDS = decltype(pds_c)::value;
    static bool attr = false;
    if (!attr) {
      (void)hipFuncSetAttribute((const void*)k_bwd_state<T, KD, C, E, PDS>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
      attr = true;
    }
    hipLaunchKernelGGL((k_bwd_state<T, KD, C, E, PDS>), dim3(s.NH * s.Nc), dim3(STATE_NTHR), smem,
                       st, s, in, dO, p, sv, bb);
    return hipGetLastError();
  };
  if (sizeof(T) == 2 && bb.dSck_lo) return go(std::integral_constant<bool, sizeof(T) == 2>{});
  return go(std::integral_constant<bool, false>{});
}

template <typename T, int KD, int C, int E>
static hipError_t chunk_inst(const Shape& s, const FwdIn& in, const void* dO, const PrepBufs& p,
                             const SavedBufs& sv,
                             const BwdBufs& bb, void* dq, void* dk, void* dv, void* dq2, void* dk2,
                             float* dg, float* dbeta, hipStream_t st) {
  const size_t smem = sizeof(ChunkSmem<T, KD, C, E>);
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)k_bwd_chunk<T, KD, C, E>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    attr = true;
  }
  hipLaunchKernelGGL((k_bwd_chunk<T, KD, C, E>), dim3(s.NH * s.Nc), dim3(CHUNK_NTHR), smem, st, s, in, dO,
                     p, sv, bb, dq, dk, dv, dq2, dk2, dg, dbeta);
  return hipGetLastError();
}

#define TLA_BWD_DISPATCH(KD_, C_, E_, CALL)              \
  if (s.K == KD_ && s.C == C_ && s.E == E_) {            \
    if (s.in_bf16) return CALL(bf16_t, KD_, C_, E_);     \
    return CALL(float, KD_, C_, E_);                     \
  }
#define TLA_BWD_FOR_EACH(CALL)      \
  TLA_BWD_DISPATCH(16, 16, 1, CALL) \
  TLA_BWD_DISPATCH(16, 16, 2, CALL) \
  TLA_BWD_DISPATCH(16, 16, 4, CALL) \
  TLA_BWD_DISPATCH(16, 16, 8, CALL) \
  TLA_BWD_DISPATCH(16, 16, 16, CALL) \
  TLA_BWD_DISPATCH(32, 32, 4, CALL) \
  TLA_BWD_DISPATCH(64, 32, 8, CALL) \
  TLA_BWD_DISPATCH(64, 64, 16, CALL) \
  TLA_BWD_DISPATCH(32, 32, 32, CALL) \
  TLA_BWD_DISPATCH(128, 64, 1, CALL) \
  TLA_BWD_DISPATCH(128, 64, 4, CALL) \
  TLA_BWD_DISPATCH(128, 64, 8, CALL) \
  TLA_BWD_DISPATCH(128, 64, 16, CALL) \
  TLA_BWD_DISPATCH(128, 32, 8, CALL)

template <typename T, int KD, int C, int E>
static bool bwd_fits_inst() {
  return sizeof(RecSmem<T, KD, C, E, bwd_waves<E>()>) <= 160 * 1024 &&
         sizeof(StateSmem<T, KD, C, E>) <= 160 * 1024 &&
         sizeof(ChunkSmem<T, KD, C, E>) <= 160 * 1024;
}

bool bwd_fits_lds(int K, int C, int E, bool bf16) {
  const Shape s{0, 1, 1, 1, K, 16, E, C, 1, 1, bf16 ? 1 : 0, 0, 0};
#define FITS_B(T_, KD_, C_, E_) bwd_fits_inst<T_, KD_, C_, E_>()
  TLA_BWD_FOR_EACH(FITS_B)
#undef FITS_B
  return false;
}

hipError_t launch_bwd_rec(const Shape& s, const FwdIn& in, const void* dO, const float* dS_final,
                          const PrepBufs& p, const BwdBufs& bb, float* ds0, hipStream_t st) {
#define CALL_REC(T_, KD_, C_, E_) rec_inst<T_, KD_, C_, E_>(s, in, dO, dS_final, p, bb, ds0, st)
  TLA_BWD_FOR_EACH(CALL_REC)
#undef CALL_REC
  return hipErrorInvalidValue;
}

hipError_t launch_bwd_state(const Shape& s, const FwdIn& in, const void* dO, const PrepBufs& p,
                            const SavedBufs& sv, const BwdBufs& bb, hipStream_t st) {
#define CALL_ST(T_, KD_, C_, E_) state_inst<T_, KD_, C_, E_>(s, in, dO, p, sv, bb, st)
  TLA_BWD_FOR_EACH(CALL_ST)
#undef CALL_ST
  return hipErrorInvalidValue;
}

hipError_t launch_bwd_chunk(const Shape& s, const FwdIn& in, const void* dO, const PrepBufs& p,
                            const SavedBufs& sv, const BwdBufs& bb, void* dq, void* dk, void* dv,
                            void* dq2, void* dk2, float* dg, float* dbeta, hipStream_t st) {
#define CALL_CH(T_, KD_, C_, E_) \
  chunk_inst<T_, KD_, C_, E_>(s, in, dO, p, sv, bb, dq, dk, dv, dq2, dk2, dg, dbeta, st)
  TLA_BWD_FOR_EACH(CALL_CH)
#undef CALL_CH
  return hipErrorInvalidValue;
}

}  // namespace tla
