// The mixer's input projection with its epilogue fused (section "Input
// projections", Alg. 2), and the plain GEMMs and transposes of its backward.
//
// Forward: y = u Wp^T, one GEMM over d_model that yields the channels of q,
// k, v, q' and k' of every head, followed in the same kernel by the causal
// depthwise convolution, SiLU / softplus and the Euclidean normalisations of
// the input side.  y therefore never makes a round trip through HBM; a
// training forward may still write it (bf16) for the backward.
//
// GEMM tiles: bf16 operands, fp32 accumulation on v_mfma_f32_32x32x16_bf16.
// A workgroup of eight waves (two per SIMD) computes 256 rows by 128 columns;
// wave (mi, ni) owns rows 64 mi .. 64 mi + 63 and columns 64 ni .. 64 ni + 63
// (2 x 2 accumulator tiles of 32 x 32; per 32-deep step 4 + 4 fragment reads
// feed 8 MFMAs).  The 32 x 32 shape and the second wave per SIMD both matter:
// measured on the device, back-to-back 16x16x32 MFMAs from a single wave
// reach about 59% of the matrix cores' rate, 32x32x16 ones 95-97%, and a
// copy instruction holds up the wave that issues it, which the SIMD's other
// wave covers.  The projection tile is 256 consecutive tokens of one batch
// row plus 16 rows above them, whose last W - 1 the convolution reads:
// recomputed rather than taken from the neighbouring tile (6% more MFMA
// work, no wait between workgroups) on 16x16x32 MFMAs, one 16-column halo
// tile per wave.  The contraction runs in stages of 64 through a ring of
// three shared-memory buffers, filled by direct global-to-LDS copies two
// stages ahead.  Rows past an operand's end are copied from clamped
// addresses and never stored; a partial last stage has its chunks past the
// contraction length zeroed in shared memory.  LDS rows are XOR-swizzled in
// 16-byte chunks, so fragment reads are free of bank conflicts while whole
// 1 KiB copies still fill them.
//
// Projection epilogue: the fp32 accumulators go through shared memory (the
// stage buffers' space); a thread then walks a run of 8 tokens for eight
// channels, keeping the last W - 1 inputs in registers, applies the taps, the
// activation and the norm (a sum over the K / 8 or E / 8 lanes of the head,
// all inside one 16-lane row group since a tile holds whole heads), and writes
// 16 bytes per token and output.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "tla_common.hpp"
#include "tla_input_side.hpp"
#include "tla_internal.hpp"

namespace tla {

constexpr int GM_NW = 8;      // waves: two per SIMD, 4 (rows) x 2 (columns)
constexpr int GM_NTHR = GM_NW * 64;
constexpr int GM_BM = 256;    // rows of a tile (tokens of a projection tile)
constexpr int GM_BN = 128;    // columns of a tile (channels of a projection tile)
constexpr int GM_BK = 64;     // contraction depth of a stage
constexpr int GM_NS = 3;      // stages in the shared-memory ring
constexpr int PJ_HALO = 16;   // rows above a projection tile
constexpr int PJ_YLD = GM_BN + 8;  // fp32 row pitch of the epilogue tile: the two lane halves of
                                   // an accumulator store (4 rows apart) hit disjoint banks

template <int HALO>
struct GemmRing {
  static constexpr int RA = GM_BM + HALO;
  typedef SwzTile<bf16_t, RA, GM_BK> TA;
  typedef SwzTile<bf16_t, GM_BN, GM_BK> TB;
  TA a[GM_NS];
  TB b[GM_NS];
  // 1 KiB copies per stage, and per wave (round-robin over the eight waves)
  static constexpr int NBA = TA::NCHK / 64, NBB = TB::NCHK / 64;
  static constexpr int MA = (NBA + GM_NW - 1) / GM_NW, MB = NBB / GM_NW;
  static_assert(TA::NCHK % 64 == 0 && NBB % GM_NW == 0, "whole 1 KiB copies");
};

struct ProjSmem {
  union {
    GemmRing<PJ_HALO> ring;
    float y[GM_BM + PJ_HALO][PJ_YLD];
  };
};
static_assert(sizeof(ProjSmem) <= 160 * 1024, "projection tile exceeds shared memory");
static_assert(sizeof(GemmRing<0>) <= 160 * 1024, "GEMM ring exceeds shared memory");

// The logical chunk a lane copies is the same in every 1 KiB block of a wave:
// physical chunk p = 64 blk + lane holds row r = p / 8, chunk (p % 8) ^ sw(r)
// with sw(r) = (r / 2) % 8, and blk = wave + 8 i keeps (r / 2) % 8 fixed.
__device__ __forceinline__ int copy_chunk(int wv, int lane) {
  return (lane & 7) ^ ((4 * (wv & 1) + (lane >> 4)) & 7);
}
__device__ __forceinline__ int copy_row(int wv, int i, int lane) {
  return 8 * (wv + GM_NW * i) + (lane >> 3);
}

// Issue the copies of the stage starting at contraction index k0 into ring
// slot `slot`; ra / rb are the lanes' row byte offsets from the bases.
template <int HALO>
__device__ __forceinline__ void issue_stage(GemmRing<HALO>& R, int slot, const bf16_t* baseA,
                                            const bf16_t* baseB,
                                            const uint32_t (&ra)[GemmRing<HALO>::MA],
                                            const uint32_t (&rb)[GemmRing<HALO>::MB], int wv,
                                            int chunk, int k0, int K) {
  typedef GemmRing<HALO> RG;
  const uint32_t kb = 2u * (uint32_t)min(k0 + 8 * chunk, K - 8);
  const uint32_t la = lds_addr(R.a[slot].d), lb = lds_addr(R.b[slot].d);
#pragma unroll
  for (int i = 0; i < RG::MA; ++i) {
    const int blk = wv + GM_NW * i;
    if (RG::NBA % GM_NW != 0 && blk >= RG::NBA) break;  // wave-uniform
    lds_dma<16>(baseA, ra[i] + kb, la + 1024 * blk);
  }
#pragma unroll
  for (int i = 0; i < RG::MB; ++i) lds_dma<16>(baseB, rb[i] + kb, lb + 1024 * (wv + GM_NW * i));
}

// Zero the chunks at contraction index K and beyond of a partial stage.
template <int HALO>
__device__ __forceinline__ void zero_tail(GemmRing<HALO>& R, int slot, int k0, int K) {
  typedef GemmRing<HALO> RG;
  for (int p = threadIdx.x; p < RG::TA::NCHK + RG::TB::NCHK; p += GM_NTHR) {
    const bool isa = p < RG::TA::NCHK;
    const int pp = isa ? p : p - RG::TA::NCHK;
    int r, c;
    RG::TA::logical(pp, r, c);  // the same chunk map for both tiles (eight chunks per row)
    if (k0 + 8 * c >= K) {
      char* d = isa ? (char*)R.a[slot].d : (char*)R.b[slot].d;
      *(uint4*)(d + 16 * pp) = make_uint4(0, 0, 0, 0);
    }
  }
}

// A wave's operand fragments of one 32-deep step, as two 16-deep halves of
// v_mfma_f32_32x32x16_bf16 operands: its 2 row tiles and 2 column tiles of 32
// (lane l holds row / column l % 32, contraction 8 (l / 32) .. + 7 of the
// half); with a halo, the halo's 16-row A fragment and the B fragment of the
// wave's halo column tile of 16, for v_mfma_f32_16x16x32_bf16 (lane l holds
// row / column l % 16, contraction 8 (l / 16) .. + 7).
struct StepFrags {
  bf16x8 a[2][2], b[2][2], ha, hb;
};

// Read step `st` (0 or 1) of the stage in ring slot `slot` into F.  Wave (mi,
// ni) owns rows 64 mi .. 64 mi + 63 and columns 64 ni .. 64 ni + 63 of the
// tile, and the halo's columns 16 (4 ni + mi) .. + 15.
template <int HALO>
__device__ __forceinline__ void read_step(const GemmRing<HALO>& R, int slot, int st, int mi, int ni,
                                          int lane, StepFrags& F) {
  const int r32 = lane & 31;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int col = 8 * (4 * st + 2 * h + (lane >> 5));
#pragma unroll
    for (int i = 0; i < 2; ++i)
      F.a[h][i] = *(const bf16x8*)R.a[slot].at(HALO + 64 * mi + 32 * i + r32, col);
#pragma unroll
    for (int j = 0; j < 2; ++j) F.b[h][j] = *(const bf16x8*)R.b[slot].at(64 * ni + 32 * j + r32, col);
  }
  if constexpr (HALO > 0) {
    const int r16 = lane & 15, col = 8 * (4 * st + (lane >> 4));
    F.ha = *(const bf16x8*)R.a[slot].at(r16, col);
    F.hb = *(const bf16x8*)R.b[slot].at(16 * (4 * ni + mi) + r16, col);
  }
}

// A compile-time loop: f(std::integral_constant<int, I>) for I = B .. E - 1.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Copy number C (0 .. MA + MB - 1) of this wave's share of a stage: A blocks
// wv, wv + 4, ... then B blocks wv, wv + 4, ...; a wave with fewer A blocks
// than MA skips the missing ones.  kb is the byte offset of the lane's chunk
// within the stage's rows.
template <int HALO, int C>
__device__ __forceinline__ void stage_copy(GemmRing<HALO>& R, int slot, const bf16_t* baseA,
                                           const bf16_t* baseB,
                                           const uint32_t (&ra)[GemmRing<HALO>::MA],
                                           const uint32_t (&rb)[GemmRing<HALO>::MB], int wv,
                                           uint32_t kb) {
  typedef GemmRing<HALO> RG;
  if constexpr (C < RG::MA) {
    const int blk = wv + GM_NW * C;
    if (RG::NBA % GM_NW != 0 && blk >= RG::NBA) return;  // wave-uniform
    lds_dma<16>(baseA, ra[C] + kb, lds_addr(R.a[slot].d) + 1024 * blk);
  } else {
    lds_dma<16>(baseB, rb[C - RG::MA] + kb,
                lds_addr(R.b[slot].d) + 1024 * (wv + GM_NW * (C - RG::MA)));
  }
}

// The products of one step: the wave's 2 x 2 tiles of 32 x 32 and, with a
// halo, its halo tile of 16 x 16 (rows 0..15, columns 16 (4 ni + mi)).
// Copies C0 .. C1 - 1 of a later stage into ring slot `slot` are issued
// spread over the 8 MFMAs (a copy instruction holds up the wave that issues
// it for about 85 cycles; between products, and with the SIMD's other wave
// issuing its own, that time overlaps the matrix core's work).
template <int HALO, int C0, int C1>
__device__ __forceinline__ void mma_step(const StepFrags& F, f32x16 (&acc)[2][2], f32x4& acch,
                                         GemmRing<HALO>& R, int slot, const bf16_t* baseA,
                                         const bf16_t* baseB,
                                         const uint32_t (&ra)[GemmRing<HALO>::MA],
                                         const uint32_t (&rb)[GemmRing<HALO>::MB], int wv,
                                         uint32_t kb) {
  static_for<0, 8>([&](auto m) {
    constexpr int M = decltype(m)::value, h = M / 4, i = (M / 2) % 2, j = M % 2;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.a[h][i], F.b[h][j], acc[i][j], 0, 0, 0);
    static_for<C0, C1>([&](auto c) {
      constexpr int C = decltype(c)::value;
      if constexpr ((C - C0) * 8 / (C1 - C0) == M) {  // copy C after product M
        stage_copy<HALO, C>(R, slot, baseA, baseB, ra, rb, wv, kb);
        __builtin_amdgcn_sched_barrier(0);
      }
    });
  });
  if constexpr (HALO > 0) acch = __builtin_amdgcn_mfma_f32_16x16x32_bf16(F.ha, F.hb, acch, 0, 0, 0);
}

// The contraction over stages [s0, s1) of 64 (K the full length), software
// pipelined by 32-deep steps.  Stage s sits in ring slot s % 3.  X holds the
// fragments of a stage's first step and Y of its second: the products of
// (s, 0) run while (s, 1) is read, and the products of (s, 1) while
// (s + 1, 0) is read, so with one wave per SIMD the shared-memory reads hide
// under the MFMAs instead of preceding them.  Before reading stage s + 1
// every wave waits for its own copies of it and the barrier makes all of
// them visible (the barrier waits for the wave's shared-memory reads, not
// for its copies); it also certifies that every wave has read stage s into
// registers, so slot s % 3 is refilled with stage s + 3 (copies run two
// stages ahead): its first CS copies under the products of (s, 1), the
// rest under those of (s + 1, 0), all before the wait for stage s + 2.  The
// waits count copies with immediates: in the steady state one stage's
// copies may stay in flight (counted as the fewest any wave issues, so a
// wave that issues one more waits a little longer), otherwise none.  A
// partial last stage has its chunks past K zeroed before it is read.
template <int HALO>
__device__ __forceinline__ void gemm_mainloop(GemmRing<HALO>& R, const bf16_t* baseA,
                                              const bf16_t* baseB,
                                              const uint32_t (&ra)[GemmRing<HALO>::MA],
                                              const uint32_t (&rb)[GemmRing<HALO>::MB], int K,
                                              int s0, int s1, f32x16 (&acc)[2][2],
                                              f32x4& acch) {
  typedef GemmRing<HALO> RG;
  static_assert(GM_NS == 3, "the waits below assume one stage in flight beyond the next");
  constexpr int MINPER = RG::NBA / GM_NW + RG::MB;  // copies per stage of the wave with the fewest
  constexpr int NC = RG::MA + RG::MB, CS = 4;       // copies per stage (at most); the first CS early
  static_assert(MINPER <= 63 && CS < NC, "copy split");
  const int wv = wave_id(), lane = lane_id();
  const int mi = wv >> 1, ni = wv & 1;
  const int chunk = copy_chunk(wv, lane);
  const int ns = s1 - s0;
  if (ns <= 0) return;
  auto kbyte = [&](int s) { return 2u * (uint32_t)min((s0 + s) * GM_BK + 8 * chunk, K - 8); };
  // make stage s visible to every wave (own copies landed, barrier), then the
  // tail of a partial stage zeroed; `more` says whether stage s + 1 has been
  // issued and may stay in flight
  auto arrive = [&](int s, bool more) {
    if (more)
      wait_vmcnt<MINPER>();
    else
      wait_vmcnt<0>();
    __syncthreads();
    const int k0 = (s0 + s) * GM_BK;
    if (k0 + GM_BK > K) {  // uniform
      zero_tail<HALO>(R, s % GM_NS, k0, K);
      __syncthreads();
    }
  };
#pragma unroll
  for (int s = 0; s < GM_NS; ++s)
    if (s < ns) issue_stage<HALO>(R, s, baseA, baseB, ra, rb, wv, chunk, (s0 + s) * GM_BK, K);
  arrive(0, ns > 1);
  StepFrags X, Y;
  read_step<HALO>(R, 0, 0, mi, ni, lane, X);
  // one stage: XC adds the late copies of stage s + 2 under (s, 0), YC the
  // early copies of stage s + 3 under (s, 1)
  auto body = [&](int s, auto xc, auto yc) {
    constexpr bool XC = decltype(xc)::value, YC = decltype(yc)::value;
    read_step<HALO>(R, s % GM_NS, 1, mi, ni, lane, Y);
    __builtin_amdgcn_sched_barrier(0);
    mma_step<HALO, CS, XC ? NC : CS>(X, acc, acch, R, (s + 2) % GM_NS, baseA, baseB, ra, rb, wv,
                                     XC ? kbyte(s + 2) : 0u);
    __builtin_amdgcn_sched_barrier(0);
    if (s + 1 < ns) {
      arrive(s + 1, s + 2 < ns);
      read_step<HALO>(R, (s + 1) % GM_NS, 0, mi, ni, lane, X);
    }
    __builtin_amdgcn_sched_barrier(0);
    mma_step<HALO, 0, YC ? CS : 0>(Y, acc, acch, R, s % GM_NS, baseA, baseB, ra, rb, wv,
                                   YC ? kbyte(s + GM_NS) : 0u);
  };
  typedef std::true_type Y_;
  typedef std::false_type N_;
  if (ns > GM_NS)
    body(0, N_{}, Y_{});  // stage 2 came whole with the prologue
  else
    body(0, N_{}, N_{});
  int s = 1;
  for (; s + GM_NS < ns; ++s) body(s, Y_{}, Y_{});
  if (s + GM_NS - 1 < ns) body(s++, Y_{}, N_{});  // the last stage's late copies
  for (; s < ns; ++s) body(s, N_{}, N_{});
}

// Tile order.  The eight accelerator dies receive workgroups round-robin and
// each has its own L2.  When the row-tile count splits evenly over the dies,
// die x takes row tiles [x n / 8, (x + 1) n / 8) and walks them in groups of
// up to four row tiles by every column tile, row tiles fastest: the 32
// workgroups a die runs at once then share each row tile's A rows eight ways
// and each column tile's B rows four ways in its L2.  Otherwise the same
// grouping runs over the whole grid.
__device__ __forceinline__ void tile_order(int bid, int nm, int nn, int& mt, int& nt) {
  int m0 = 0, per = nm, j = bid;
  if ((nm & 7) == 0) {
    per = nm >> 3;
    m0 = (bid & 7) * per;
    j = bid >> 3;
  }
  const int gm = (per % 4 == 0) ? 4 : (per % 2 == 0) ? 2 : 1;
  const int grp = j / (gm * nn), r = j % (gm * nn);
  mt = m0 + grp * gm + r % gm;
  nt = r / gm;
}

// ------------------------------------------------------------ fused forward
template <int W>
__global__ __launch_bounds__(GM_NTHR) void k_proj_in(ProjArgs a, const bf16_t* __restrict__ u,
                                                     const bf16_t* __restrict__ Wp,
                                                     const float* __restrict__ w, bf16_t* q,
                                                     bf16_t* k, bf16_t* v, bf16_t* q2, bf16_t* k2,
                                                     bf16_t* ysave) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  ProjSmem& sm = *reinterpret_cast<ProjSmem*>(smem_raw);
  typedef GemmRing<PJ_HALO> RG;
  const int wv = wave_id(), lane = lane_id();

  int mt, ct;
  tile_order(blockIdx.x, a.n_mt, a.n_ct, mt, ct);
  const int b = mt / a.tiles_per_row, t0 = (mt % a.tiles_per_row) * GM_BM, n0 = ct * GM_BN;
  const int tbase = max(t0 - PJ_HALO, 0);
  const bf16_t* baseA = uniform_ptr(u + ((size_t)b * a.T + tbase) * a.Dm);
  const bf16_t* baseB = uniform_ptr(Wp + (size_t)n0 * a.Dm);
  uint32_t ra[RG::MA], rb[RG::MB];
#pragma unroll
  for (int i = 0; i < RG::MA; ++i) {
    const int t = min(max(t0 - PJ_HALO + copy_row(wv, i, lane), 0), a.T - 1);
    ra[i] = (uint32_t)(t - tbase) * (uint32_t)a.Dm * 2u;
  }
#pragma unroll
  for (int i = 0; i < RG::MB; ++i) {
    const int c = min(n0 + copy_row(wv, i, lane), a.Ctot - 1);
    rb[i] = (uint32_t)(c - n0) * (uint32_t)a.Dm * 2u;
  }
  f32x16 acc[2][2];
  f32x4 acch = zero4();
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  gemm_mainloop<PJ_HALO>(sm.ring, baseA, baseB, ra, rb, a.Dm, 0, (a.Dm + GM_BK - 1) / GM_BK, acc,
                         acch);

  // accumulators -> fp32 tile (row = 16 + token - t0, column = channel - n0)
  __syncthreads();  // every wave is done with the ring
  {
    // 32 x 32 tile (i, j): register r of lane l holds row 8 (r / 4) + 4 (l / 32)
    // + r % 4, column l % 32; 16 x 16 halo tile: register r of lane l holds
    // row 4 (l / 16) + r, column l % 16
    const int mi = wv >> 1, ni = wv & 1;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sm.y[PJ_HALO + 64 * mi + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)]
              [64 * ni + 32 * j + (lane & 31)] = acc[i][j][r];
#pragma unroll
    for (int r = 0; r < 4; ++r)
      sm.y[4 * (lane >> 4) + r][16 * (4 * ni + mi) + (lane & 15)] = acch[r];
  }
  __syncthreads();

  // epilogue: thread = 8 channels (16 lanes per token) x a run of PJ_RUN tokens
  constexpr int PJ_RUN = GM_BM / (GM_NTHR / 16);
  const int cl = threadIdx.x & 15, run = threadIdx.x >> 4;
  const int c = n0 + 8 * cl;
  const bool on_c = c < a.Ctot;
  const int cc = on_c ? c : a.Ctot - 8;  // lanes past the channels compute (and never store) the last ones
  const ConvLane L = conv_lane(a, cc);
  const bool silu = L.kind <= 2;
  bf16_t* out = pick(L.kind, q, k, v, q2, k2) + (size_t)b * a.T * a.H * L.width + L.off;
  const size_t orow = (size_t)a.H * L.width;
  float wt[W][8];
#pragma unroll
  for (int j = 0; j < W; ++j) {
    const f32x4 x0 = *(const f32x4*)(w + (size_t)j * a.Ctot + cc);
    const f32x4 x1 = *(const f32x4*)(w + (size_t)j * a.Ctot + cc + 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      wt[j][i] = x0[i];
      wt[j][4 + i] = x1[i];
    }
  }
  const int r0 = PJ_RUN * run;
  float hist[W > 1 ? W - 1 : 1][8];
#pragma unroll
  for (int h = 0; h < W - 1; ++h) {
    const float* yr = &sm.y[PJ_HALO + r0 - 1 - h][8 * cl];
    const bool live = t0 + r0 - 1 - h >= 0;  // tokens before the row's start count as zero
#pragma unroll
    for (int i = 0; i < 8; ++i) hist[h][i] = live ? yr[i] : 0.f;
  }
  bf16_t* yout = ysave ? ysave + (size_t)b * a.T * a.Ctot + c : nullptr;
  for (int rr = 0; rr < PJ_RUN; ++rr) {
    const int t = t0 + r0 + rr;
    float x[8], z[8], r[8], ss = 0.f;
    const float* yr = &sm.y[PJ_HALO + r0 + rr][8 * cl];
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = yr[i];
    conv8<W>(wt, hist, x, z);
    push_hist<W>(hist, x);
    act8(silu, z, r);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += r[i] * r[i];
    ss = lane_group_sum(ss, L.lpr);  // every lane of the wave takes part
    if (L.lpr) {
      const float inv = rsqrtf(ss + a.eps);
#pragma unroll
      for (int i = 0; i < 8; ++i) r[i] *= inv;
    }
    if (on_c && t < a.T) {
      store8(out + (size_t)t * orow, r);
      if (yout) store8(yout + (size_t)t * a.Ctot, x);
    }
  }
}

ProjArgs proj_args(int B, int T, int Dm, int H, int K, int V, int E, int W, float eps) {
  ProjArgs a;
  a.B = B, a.T = T, a.Dm = Dm, a.H = H, a.K = K, a.V = V, a.E = E, a.W = W;
  a.Ctot = H * (2 * K + V + 2 * E);
  a.tiles_per_row = (T + GM_BM - 1) / GM_BM;
  a.n_mt = B * a.tiles_per_row;
  a.n_ct = (a.Ctot + GM_BN - 1) / GM_BN;
  a.eps = eps;
  return a;
}

hipError_t launch_proj_in(const ProjArgs& a, const void* u, const void* Wp, const float* w,
                          void* const* out, void* y, hipStream_t st) {
  const unsigned nblk = (unsigned)a.n_mt * (unsigned)a.n_ct;
  if (nblk == 0) return hipSuccess;
  const size_t smem = sizeof(ProjSmem);
#define PROJ_L(W_)                                                                               \
  case W_:                                                                                       \
    (void)hipFuncSetAttribute((const void*)k_proj_in<W_>,                                        \
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);            \
    hipLaunchKernelGGL((k_proj_in<W_>), dim3(nblk), dim3(GM_NTHR), smem, st, a, (const bf16_t*)u, \
                       (const bf16_t*)Wp, w, (bf16_t*)out[0], (bf16_t*)out[1], (bf16_t*)out[2],   \
                       (bf16_t*)out[3], (bf16_t*)out[4], (bf16_t*)y);                            \
    break;
  switch (a.W) {
    PROJ_L(1) PROJ_L(2) PROJ_L(3) PROJ_L(4)
    default: return hipErrorInvalidValue;
  }
#undef PROJ_L
  return hipGetLastError();
}

// --------------------------------------------------------------- plain GEMM
// C[M][N] = A[M][K] B[N][K]^T over the stages of split blockIdx.y.
template <bool OUT_BF16>
__global__ __launch_bounds__(GM_NTHR) void k_gemm_nt(long long M, long long N, int K,
                                                     const bf16_t* __restrict__ A,
                                                     const bf16_t* __restrict__ Bm, void* C,
                                                     long long ldc, int splits, float* part) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  typedef GemmRing<0> RG;
  RG& R = *reinterpret_cast<RG*>(smem_raw);
  const int wv = wave_id(), lane = lane_id();
  int mti, nti;
  tile_order(blockIdx.x, (int)((M + GM_BM - 1) / GM_BM), (int)((N + GM_BN - 1) / GM_BN), mti, nti);
  const long long m0 = (long long)mti * GM_BM, n0 = (long long)nti * GM_BN;
  const bf16_t* baseA = uniform_ptr(A + m0 * K);
  const bf16_t* baseB = uniform_ptr(Bm + n0 * K);
  uint32_t ra[RG::MA], rb[RG::MB];
#pragma unroll
  for (int i = 0; i < RG::MA; ++i)
    ra[i] = (uint32_t)(min(m0 + copy_row(wv, i, lane), M - 1) - m0) * (uint32_t)K * 2u;
#pragma unroll
  for (int i = 0; i < RG::MB; ++i)
    rb[i] = (uint32_t)(min(n0 + copy_row(wv, i, lane), N - 1) - n0) * (uint32_t)K * 2u;
  const int nst = (K + GM_BK - 1) / GM_BK, z = blockIdx.y;
  const int s0 = (int)((long long)nst * z / splits), s1 = (int)((long long)nst * (z + 1) / splits);
  f32x16 acc[2][2];
  f32x4 acch = zero4();
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  gemm_mainloop<0>(R, baseA, baseB, ra, rb, K, s0, s1, acc, acch);

  // registers 4 q .. 4 q + 3 of lane l in tile (i, j) hold rows 8 q + 4 (l / 32)
  // + 0..3, column l % 32; after the quad transpose (lanes 4 m .. 4 m + 3
  // exchange) lane l holds row 8 q + 4 (l / 32) + l % 4, columns
  // 4 ((l % 32) / 4) .. + 3
  const int mi = wv >> 1, ni = wv & 1, n = lane & 31;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 x = quad_transpose(f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                           acc[i][j][4 * q + 3]}, n);
      const long long row = m0 + 64 * mi + 32 * i + 8 * q + 4 * (lane >> 5) + (n & 3);
      const long long col = n0 + 64 * ni + 32 * j + 4 * (n >> 2);
      if (row < M && col < N) {  // N is a multiple of 4
        if (splits > 1) {
          *(f32x4*)(part + ((long long)z * M + row) * N + col) = x;
        } else if constexpr (OUT_BF16) {
          *(u32x2*)((bf16_t*)C + row * ldc + col) = __builtin_bit_cast(u32x2, cvt_frag<bf16_t>(x));
        } else {
          *(f32x4*)((float*)C + row * ldc + col) = x;
        }
      }
    }
}

// C = sum over splits of the partial products, in split order
template <bool OUT_BF16>
__global__ __launch_bounds__(256) void k_sum_splits(long long M, long long N, int splits,
                                                    const float* __restrict__ part, void* C,
                                                    long long ldc) {
  const long long i4 = (long long)blockIdx.x * 256 + threadIdx.x;  // index of 4 columns
  const long long nq = N / 4;
  if (i4 >= M * nq) return;
  const long long row = i4 / nq, col = 4 * (i4 % nq);
  f32x4 s = *(const f32x4*)(part + row * N + col);
  for (int z = 1; z < splits; ++z) s += *(const f32x4*)(part + ((long long)z * M + row) * N + col);
  if constexpr (OUT_BF16)
    *(u32x2*)((bf16_t*)C + row * ldc + col) = __builtin_bit_cast(u32x2, cvt_frag<bf16_t>(s));
  else
    *(f32x4*)((float*)C + row * ldc + col) = s;
}

int gemm_splits(long long M, long long N, long long K) {
  const long long tiles = ((M + GM_BM - 1) / GM_BM) * ((N + GM_BN - 1) / GM_BN);
  const long long nst = (K + GM_BK - 1) / GM_BK;
  // fill the 256 compute units in whole rounds of one tile each, with at
  // least eight stages per split
  int best = 1;
  double best_eff = 0.0;
  for (int s = 1; s <= 8 && nst / s >= 8; ++s) {
    const long long work = tiles * s;
    const double eff = (double)work / (double)(((work + 255) / 256) * 256);
    if (eff > best_eff + 0.05) best = s, best_eff = eff;
  }
  return best;
}

hipError_t launch_gemm_nt(long long M, long long N, long long K, const void* A, const void* Bm,
                          void* C, bool c_bf16, long long ldc, int splits, float* part,
                          hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const long long tiles = ((M + GM_BM - 1) / GM_BM) * ((N + GM_BN - 1) / GM_BN);
  const size_t smem = sizeof(GemmRing<0>);
  const dim3 grid((unsigned)tiles, (unsigned)splits);
  if (c_bf16) {
    (void)hipFuncSetAttribute((const void*)k_gemm_nt<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)smem);
    hipLaunchKernelGGL(k_gemm_nt<true>, grid, dim3(GM_NTHR), smem, st, M, N, (int)K,
                       (const bf16_t*)A, (const bf16_t*)Bm, C, ldc, splits, part);
  } else {
    (void)hipFuncSetAttribute((const void*)k_gemm_nt<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)smem);
    hipLaunchKernelGGL(k_gemm_nt<false>, grid, dim3(GM_NTHR), smem, st, M, N, (int)K,
                       (const bf16_t*)A, (const bf16_t*)Bm, C, ldc, splits, part);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const long long n4 = M * (N / 4);
  const unsigned nb = (unsigned)((n4 + 255) / 256);
  if (c_bf16)
    hipLaunchKernelGGL(k_sum_splits<true>, dim3(nb), dim3(256), 0, st, M, N, splits, part, C, ldc);
  else
    hipLaunchKernelGGL(k_sum_splits<false>, dim3(nb), dim3(256), 0, st, M, N, splits, part, C, ldc);
  return hipGetLastError();
}

// ---------------------------------------------------------------- transpose
// out [C][Rp] = in [R][C]^T for 64 x 64 tiles through shared memory; rows R ..
// Rp - 1 of the result are zero.  C is a multiple of 8.
__global__ __launch_bounds__(256) void k_transpose(long long R, long long C, long long Rp,
                                                   const bf16_t* __restrict__ in,
                                                   bf16_t* __restrict__ out) {
  __shared__ bf16_t tile[64][64 + 2];
  const long long r0 = (long long)blockIdx.x * 64, c0 = (long long)blockIdx.y * 64;
  // load: 64 rows x 8 chunks of 8 elements, two chunks per thread
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int idx = threadIdx.x + 256 * h, rr = idx >> 3, ch = idx & 7;
    const long long r = r0 + rr, c = c0 + 8 * ch;
    uint4 x = make_uint4(0, 0, 0, 0);
    if (r < R && c < C) x = *(const uint4*)(in + r * C + c);
    const bf16_t* e = (const bf16_t*)&x;
#pragma unroll
    for (int i = 0; i < 8; ++i) tile[rr][8 * ch + i] = e[i];
  }
  __syncthreads();
  // store: 64 result rows (columns of in) x 8 chunks of 8 elements
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int idx = threadIdx.x + 256 * h, cc = idx >> 3, ch = idx & 7;
    const long long c = c0 + cc, r = r0 + 8 * ch;
    if (c >= C || r >= Rp) continue;
    bf16_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = tile[8 * ch + i][cc];
    *(uint4*)(out + c * Rp + r) = *(const uint4*)e;
  }
}

hipError_t launch_transpose(long long R, long long C, long long Rp, const void* in, void* out,
                            hipStream_t st) {
  if (Rp <= 0 || C <= 0) return hipSuccess;
  const dim3 grid((unsigned)((Rp + 63) / 64), (unsigned)((C + 63) / 64));
  hipLaunchKernelGGL(k_transpose, grid, dim3(256), 0, st, R, C, Rp, (const bf16_t*)in,
                     (bf16_t*)out);
  return hipGetLastError();
}

}  // namespace tla
