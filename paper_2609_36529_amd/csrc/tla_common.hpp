// Device helpers shared by the triadic linear attention kernels (gfx950).
//
// Fragment convention (64-wide wavefront, 16x16 MFMA tiles):
//   lane l, group g = l / 16, index n = l % 16
//   A fragment of a 16 x 16k block: lane holds A[n][4g + j], j = 0..3
//   B fragment of a 16k x 16 block: lane holds B[4g + j][n], j = 0..3
//   accumulator (16 x 16, fp32):    lane holds C[4g + j][n], j = 0..3
// An accumulator is therefore already the B fragment of itself (its row index
// is the contraction index) and the A fragment of its transpose.  Two 16-deep
// bf16 fragments feed one v_mfma_f32_16x16x32_bf16 (slots 0..3 from the first
// block, 4..7 from the second); the contraction does not depend on how the
// hardware orders k inside an instruction as long as A and B agree.  fp32
// operands go through four v_mfma_f32_16x16x4_f32 per 16-deep block.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tla {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;  // bf16 storage in global memory
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
// The wave index, marked uniform (read from the first lane) so that branches
// on it are scalar and do not split the wave's code into exec-masked blocks.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// ---------------------------------------------------------------- scalar I/O
template <typename T> struct Elem;
template <> struct Elem<float> {
  typedef float storage;
  typedef f32x4 frag;  // 4 operand values of a 16-deep fragment
  __device__ static __forceinline__ float to_f(float x) { return x; }
  __device__ static __forceinline__ float from_f(float x) { return x; }
};
template <> struct Elem<bf16_t> {
  typedef bf16_t storage;
  typedef bf16x4 frag;
  __device__ static __forceinline__ float to_f(bf16_t x) {
    return __uint_as_float(((uint32_t)x) << 16);
  }
  __device__ static __forceinline__ bf16_t from_f(float x) {
    __bf16 b = (__bf16)x;  // round to nearest even
    return __builtin_bit_cast(bf16_t, b);
  }
};

template <typename T>
__device__ __forceinline__ float ld_f(const T* p) { return Elem<T>::to_f(*p); }

// 4 consecutive elements as floats (p aligned to 4 elements)
__device__ __forceinline__ f32x4 ld4_f(const float* p) { return *(const f32x4*)p; }
__device__ __forceinline__ f32x4 ld4_f(const bf16_t* p) {
  uint2 u = *(const uint2*)p;
  f32x4 r;
  r[0] = __uint_as_float(u.x << 16);
  r[1] = __uint_as_float(u.x & 0xffff0000u);
  r[2] = __uint_as_float(u.y << 16);
  r[3] = __uint_as_float(u.y & 0xffff0000u);
  return r;
}

// ------------------------------------------------------------- fragments
// Load a 4-element fragment from contiguous storage.
__device__ __forceinline__ f32x4 ld_frag(const float* p) { return *(const f32x4*)p; }
__device__ __forceinline__ bf16x4 ld_frag(const bf16_t* p) {
  return __builtin_bit_cast(bf16x4, *(const uint2*)p);
}

// Convert 4 fp32 values (e.g. an accumulator) into an operand fragment.
template <typename T> __device__ __forceinline__ typename Elem<T>::frag cvt_frag(f32x4 x);
template <> __device__ __forceinline__ f32x4 cvt_frag<float>(f32x4 x) { return x; }
template <> __device__ __forceinline__ bf16x4 cvt_frag<bf16_t>(f32x4 x) {
  bf16x4 r;
  r[0] = (__bf16)x[0];
  r[1] = (__bf16)x[1];
  r[2] = (__bf16)x[2];
  r[3] = (__bf16)x[3];
  return r;
}

// Split 4 fp32 values into a bf16 pair hi + lo whose sum carries ~16
// mantissa bits: hi = rne(x), lo = rne(x - hi).  Used for the fp32-computed
// operands (U, M, Tu) whose plain bf16 rounding would dominate the error.
__device__ __forceinline__ f32x4 bf16x4_to_f(bf16x4 x) {
  return f32x4{(float)x[0], (float)x[1], (float)x[2], (float)x[3]};
}
__device__ __forceinline__ f32x4 frag_to_f(bf16x4 x) { return bf16x4_to_f(x); }
__device__ __forceinline__ f32x4 frag_to_f(f32x4 x) { return x; }
__device__ __forceinline__ void split_frag(f32x4 x, bf16x4& hi, bf16x4& lo) {
  hi = cvt_frag<bf16_t>(x);
  lo = cvt_frag<bf16_t>(x - bf16x4_to_f(hi));
}
__device__ __forceinline__ void split_frag(f32x4 x, f32x4& hi, f32x4& lo) {
  hi = x;
  lo = zero4();
}

// LDS row strides are padded to (2 mod 32) dwords for bf16 rows and (4 mod
// 32) for fp32 rows (row length + 4 elements), so the 16 lanes that read one
// fragment column hit distinct banks.  Such bf16 rows are only 8-byte aligned:
// 8-element copies into them use two 8-byte stores.
template <typename T>
__device__ __forceinline__ void lds_put8(T* dst, const T* src) {
  if constexpr (sizeof(T) == 2) {
    ((uint2*)dst)[0] = ((const uint2*)src)[0];
    ((uint2*)dst)[1] = ((const uint2*)src)[1];
  } else {
    ((float4*)dst)[0] = ((const float4*)src)[0];
    ((float4*)dst)[1] = ((const float4*)src)[1];
  }
}
// Store 4 elements (a column segment of a transposed tile) with one write.
template <typename T>
__device__ __forceinline__ void lds_put4(T* dst, T a, T b, T c, T d) {
  if constexpr (sizeof(T) == 2) {
    uint2 u;
    u.x = (uint32_t)a | ((uint32_t)b << 16);
    u.y = (uint32_t)c | ((uint32_t)d << 16);
    *(uint2*)dst = u;
  } else {
    *(float4*)dst = make_float4(a, b, c, d);
  }
}

// Gather 4 strided elements into a fragment (stride in elements).
template <typename T>
__device__ __forceinline__ typename Elem<T>::frag ld_frag_strided(const T* p, int stride) {
  f32x4 x;
  x[0] = Elem<T>::to_f(p[0]);
  x[1] = Elem<T>::to_f(p[stride]);
  x[2] = Elem<T>::to_f(p[2 * stride]);
  x[3] = Elem<T>::to_f(p[3 * stride]);
  return cvt_frag<T>(x);
}

// A row of N consecutive values from shared memory (16-byte aligned when N
// fills whole 16-byte words) with the widest reads the length allows.
template <int N, typename V>
__device__ __forceinline__ void lds_row(V (&x)[N], const V* src) {
  constexpr int PER = 16 / (int)sizeof(V);  // values per 16-byte read
  if constexpr (N % PER == 0) {
#pragma unroll
    for (int i = 0; i < N / PER; ++i) {
      const uint4 w = ((const uint4*)src)[i];
      V t[PER];
      __builtin_memcpy(t, &w, 16);
#pragma unroll
      for (int k = 0; k < PER; ++k) x[PER * i + k] = t[k];
    }
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] = src[i];
  }
}

// ------------------------------------------------------------------ MFMA
__device__ __forceinline__ void mma16(f32x4& acc, f32x4 a, f32x4 b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], acc, 0, 0, 0);
}
__device__ __forceinline__ void mma16(f32x4& acc, bf16x4 a, bf16x4 b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a),
                                                  __builtin_bit_cast(i16x4, b), acc, 0, 0, 0);
}
// Two 16-deep blocks at once.
__device__ __forceinline__ void mma32(f32x4& acc, f32x4 a0, f32x4 a1, f32x4 b0, f32x4 b1) {
  mma16(acc, a0, b0);
  mma16(acc, a1, b1);
}
__device__ __forceinline__ void mma32(f32x4& acc, bf16x4 a0, bf16x4 a1, bf16x4 b0, bf16x4 b1) {
  bf16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
  bf16x8 b = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}

// A 32-deep A operand held as one piece: lane group g's eight consecutive
// contraction indices (a 16-byte read for bf16, two fp32 fragments).
template <typename T> struct Frag8;
template <> struct Frag8<bf16_t> { bf16x8 v; };
template <> struct Frag8<float> { f32x4 lo, hi; };
__device__ __forceinline__ void mma32(f32x4& acc, const Frag8<bf16_t>& a, bf16x4 b0, bf16x4 b1) {
  const bf16x8 b = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma32(f32x4& acc, const Frag8<float>& a, f32x4 b0, f32x4 b1) {
  mma16(acc, a.lo, b0);
  mma16(acc, a.hi, b1);
}

// Fast exp of a non-positive argument (every decay factor here is exp of a
// difference of accumulated log-gates that is <= 0).
__device__ __forceinline__ float exp_nonpos(float x) { return __expf(x); }

// ------------------------------------------------------------- reductions
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
// Sum over the 16 lanes that share a group g (lanes 16g .. 16g + 15), with
// DPP lane permutations (VALU, no LDS round trip): swap neighbours, swap
// pairs, mirror within each 8-lane half, mirror within the 16-lane row.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF,
                                                            0xF, true));
}
__device__ __forceinline__ float group16_sum(float x) {
  x += dpp_f<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp_f<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp_f<0x141>(x);  // row_half_mirror
  x += dpp_f<0x140>(x);  // row_mirror
  return x;
}

// X = (I + L)^{-1} for a strictly lower-triangular C x C matrix L (C a
// multiple of 16), blockwise: the 16 x 16 diagonal blocks by forward
// substitution (one column per thread), then the blocks below the diagonal
// level by level, X_IJ = -X_II sum_{K=J}^{I-1} L_IK X_KJ (all blocks of one
// level at once, one wave per block, both products on the fp32 MFMA).
// L(r, c) is an accessor; X is a C x ldx fp32 LDS array; Y is
// (C/16 - 1) x 16 x 17 floats of LDS scratch.  Every thread of the
// workgroup must call it (NTHR / 64 >= C / 16 - 1 waves); it ends with a
// barrier.
template <int C, int NTHR, typename LF>
__device__ void unit_lower_inverse(LF L, float* X, int ldx, float* Y) {
  constexpr int NT = C / 16;
  static_assert(NTHR / 64 >= NT - 1, "one wave per off-diagonal block of a level");
  const int tid = threadIdx.x;
  for (int idx = tid; idx < C * C; idx += NTHR) X[(idx / C) * ldx + idx % C] = 0.f;
  __syncthreads();
  if (tid < C) {
    const int r0 = 16 * (tid / 16), col = tid % 16;
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float acc = 0.f;
#pragma unroll
      for (int j = 0; j < i; ++j) acc += L(r0 + i, r0 + j) * x[j];
      x[i] = (i < col) ? 0.f : ((i == col) ? 1.f : -acc);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) X[(r0 + i) * ldx + r0 + col] = x[i];
  }
  __syncthreads();
  // 16x16x4 fp32 MFMA: lane (g, n) gives A[n][g] and B[g][n] of each 4-deep
  // step and holds C[4 g + j][n]
  const int w = tid >> 6, g = (tid >> 4) & 3, n = tid & 15;
  for (int d = 1; d < NT; ++d) {
    const bool act = w < NT - d;  // wave w: block (I, J) = (d + w, w)
    const int I = d + w, J = w;
    if (act) {
      f32x4 y = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int kb = 16 * J; kb < 16 * I; kb += 4)
        y = __builtin_amdgcn_mfma_f32_16x16x4f32(L(16 * I + n, kb + g), X[(kb + g) * ldx + 16 * J + n],
                                                 y, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < 4; ++j) Y[(w * 16 + 4 * g + j) * 17 + n] = y[j];
    }
    __syncthreads();
    if (act) {
      f32x4 x = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 0; m < 16; m += 4)
        x = __builtin_amdgcn_mfma_f32_16x16x4f32(X[(16 * I + n) * ldx + 16 * I + m + g],
                                                 Y[(w * 16 + m + g) * 17 + n], x, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < 4; ++j) X[(16 * I + 4 * g + j) * ldx + 16 * J + n] = -x[j];
    }
    __syncthreads();
  }
}

// 8 consecutive elements kept as raw 32-bit words, so that a prefetch load is
// not unpacked (and waited for) before the data is written to LDS.
template <typename T>
struct Raw8 {
  uint4 w[sizeof(T) / 2];  // bf16: one 16-byte word; fp32: two
  __device__ __forceinline__ T get(int i) const {
    if constexpr (sizeof(T) == 2) {
      const uint32_t d = (i < 2) ? w[0].x : (i < 4) ? w[0].y : (i < 6) ? w[0].z : w[0].w;
      return (T)((i & 1) ? (d >> 16) : (d & 0xffffu));
    } else {
      const uint4& q = w[i >> 2];
      const uint32_t d = ((i & 3) == 0) ? q.x : ((i & 3) == 1) ? q.y : ((i & 3) == 2) ? q.z : q.w;
      return __uint_as_float(d);
    }
  }
};
template <typename T>
__device__ __forceinline__ Raw8<T> load8(const T* src) {
  Raw8<T> r;
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 2); ++i) r.w[i] = ((const uint4*)src)[i];
  return r;
}
template <typename T>
__device__ __forceinline__ Raw8<T> zero_raw8() {
  Raw8<T> r;
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 2); ++i) r.w[i] = make_uint4(0, 0, 0, 0);
  return r;
}
template <typename T>
__device__ __forceinline__ void lds_put_raw8(T* dst, const Raw8<T>& r) {
  if constexpr (sizeof(T) == 2) {
    ((uint2*)dst)[0] = make_uint2(r.w[0].x, r.w[0].y);
    ((uint2*)dst)[1] = make_uint2(r.w[0].z, r.w[0].w);
  } else {
    ((uint4*)dst)[0] = r.w[0];
    ((uint4*)dst)[1] = r.w[1];
  }
}

// Loads of N consecutive 32-bit words (16- or 8-byte accesses) and element
// access into such words.
template <int N>
__device__ __forceinline__ void ld_words(uint32_t (&w)[N], const void* src) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
      const uint4 x = ((const uint4*)src)[i];
      w[4 * i] = x.x;
      w[4 * i + 1] = x.y;
      w[4 * i + 2] = x.z;
      w[4 * i + 3] = x.w;
    }
  } else {
    static_assert(N == 2, "word count");
    const uint2 x = *(const uint2*)src;
    w[0] = x.x;
    w[1] = x.y;
  }
}
template <typename T, int N>
__device__ __forceinline__ T word_elem(const uint32_t (&w)[N], int i) {
  if constexpr (sizeof(T) == 2) return (T)((i & 1) ? (w[i >> 1] >> 16) : (w[i >> 1] & 0xffffu));
  else return __uint_as_float(w[i]);
}

// 32-deep MFMA step on raw 8-element operands: lane (g, n) holds the
// contraction indices 8g .. 8g + 7 of row n of A and of column n of B (any
// assignment of the 32 indices to lanes works as long as A and B agree).
// bf16: one 16x16x32 MFMA; fp32: two 16-deep fp32 steps.
__device__ __forceinline__ void mma8(f32x4& acc, const Raw8<bf16_t>& a, const Raw8<bf16_t>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a.w[0]),
                                                __builtin_bit_cast(bf16x8, b.w[0]), acc, 0, 0, 0);
}
__device__ __forceinline__ void mma8(f32x4& acc, const Raw8<float>& a, const Raw8<float>& b) {
  mma16(acc, __builtin_bit_cast(f32x4, a.w[0]), __builtin_bit_cast(f32x4, b.w[0]));
  mma16(acc, __builtin_bit_cast(f32x4, a.w[1]), __builtin_bit_cast(f32x4, b.w[1]));
}
// The 8 values as floats.
template <typename T>
__device__ __forceinline__ void raw8_to_f(const Raw8<T>& r, float* x) {
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = Elem<T>::to_f(r.get(i));
}

// Transposed reduction over the 16 lanes of a group: every lane brings 16
// values v[0..15]; afterwards lane n (of the group) holds the sum over the 16
// lanes of v[n].  Four exchange rounds halve the live values each time (15
// lane moves instead of 64 for sixteen separate reductions).  The lane pairs
// of each round differ in the bit that decides which half a lane keeps:
// rotate by 8 (bit 3), mirror within 8 (bit 2), reverse within 4 (bit 1),
// swap neighbours (bit 0).
__device__ __forceinline__ float group16_transpose_sum(const float (&v)[16], int n) {
  float a[8], b[4], c[2];
  const bool b3 = n & 8, b2 = n & 4, b1 = n & 2, b0 = n & 1;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float send = b3 ? v[i] : v[i + 8];
    a[i] = (b3 ? v[i + 8] : v[i]) + dpp_f<0x128>(send);  // row_ror:8
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float send = b2 ? a[i] : a[i + 4];
    b[i] = (b2 ? a[i + 4] : a[i]) + dpp_f<0x141>(send);  // row_half_mirror
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float send = b1 ? b[i] : b[i + 2];
    c[i] = (b1 ? b[i + 2] : b[i]) + dpp_f<0x1B>(send);   // quad_perm [3,2,1,0]
  }
  const float send = b0 ? c[0] : c[1];
  return (b0 ? c[1] : c[0]) + dpp_f<0xB1>(send);        // quad_perm [1,0,3,2]
}

// A 16-byte chunk into shared memory at an 8-byte aligned address (padded
// rows are not 16-byte aligned): two 8-byte writes.
template <typename T>
__device__ __forceinline__ void lds_put16(T* dst, uint4 x) {
  ((uint2*)dst)[0] = make_uint2(x.x, x.y);
  ((uint2*)dst)[1] = make_uint2(x.z, x.w);
}

// Four consecutive values to global memory in the element type (one 8-byte
// store for bf16, one 16-byte store for fp32).
template <typename T>
__device__ __forceinline__ void put4(T* dst, f32x4 x) {
  if constexpr (sizeof(T) == 2)
    *(uint2*)dst = __builtin_bit_cast(uint2, cvt_frag<bf16_t>(x));
  else
    *(f32x4*)dst = x;
}

// Vector stores issued from inline assembly: exactly one instruction each, so
// a kernel can count them in an explicit vmcnt wait (on gfx9 a store counts
// in vmcnt until the write is acknowledged, in issue order with the loads).
// They carry the nontemporal hint: every use here writes data that only a
// later kernel reads (checkpoints, saved U and V - W, state gradients), so it
// should not displace the operands the workgroups of a head share in L2.
__device__ __forceinline__ void gstore_b32(void* p, uint32_t x) {
  asm volatile("global_store_dword %0, %1, off nt" ::"v"(p), "v"(x) : "memory");
}
__device__ __forceinline__ void gstore_b64(void* p, u32x2 x) {
  asm volatile("global_store_dwordx2 %0, %1, off nt" ::"v"(p), "v"(x) : "memory");
}
// (a VALU write to the data registers of a store of more than 8 bytes needs
// one wait state after it; the compiler cannot see that inside the assembly,
// so the nop is part of it)
__device__ __forceinline__ void gstore_b128(void* p, u32x4 x) {
  asm volatile("global_store_dwordx4 %0, %1, off nt\n\ts_nop 1" ::"v"(p), "v"(x) : "memory");
}

// gfx950 transposing shared-memory read (ds_read_b64_tr_b16).  Within each
// group of 16 lanes, let row s of a 16 x 4 matrix IN be the four 16-bit
// elements that lane s of the group reads at its own address p; lane o of the
// group receives IN[4 j + o / 4][o % 4] as its element j (j = 0..3).  (The
// lane layout was established on the device with an in-bounds test.)
__device__ __forceinline__ bf16x4 lds_read_tr16(const void* p) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
  const v4i16 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)const_cast<void*>(p));
  return __builtin_bit_cast(bf16x4, r);
}

// 4 x 4 transposes within each quad of lanes by two DPP exchange rounds: a
// lane (g, n) that holds rows 4 g + j (j = 0..3) of column n of a 16 x 16
// accumulator tile afterwards holds row 4 g + n % 4, columns 4 (n / 4) + j.
__device__ __forceinline__ f32x4 quad_transpose(f32x4 x, int n) {
  const int i = n & 3;
  const bool b0 = i & 1, b1 = i & 2;
  float t = dpp_f<0xB1>(b0 ? x[0] : x[1]);  // lanes differing in bit 0
  x[0] = b0 ? t : x[0];
  x[1] = b0 ? x[1] : t;
  t = dpp_f<0xB1>(b0 ? x[2] : x[3]);
  x[2] = b0 ? t : x[2];
  x[3] = b0 ? x[3] : t;
  t = dpp_f<0x4E>(b1 ? x[0] : x[2]);        // lanes differing in bit 1
  x[0] = b1 ? t : x[0];
  x[2] = b1 ? x[2] : t;
  t = dpp_f<0x4E>(b1 ? x[1] : x[3]);
  x[1] = b1 ? t : x[1];
  x[3] = b1 ? x[3] : t;
  return x;
}

// Store a 16 x 16 accumulator tile (lane (g, n) holds rows 4 g + j, column n)
// into a row-major tile at dst (row r at dst + ld r, ld = 16 by default) after
// quad_transpose: one 8-byte (bf16) or 16-byte (fp32) store per lane instead
// of four scalar ones (one store instruction per tile, countable in a vmcnt
// wait).
template <typename T>
__device__ __forceinline__ void store_tile16(T* dst, f32x4 x, int g, int n, int ld = 16) {
  x = quad_transpose(x, n);
  T* p = dst + (4 * g + (n & 3)) * ld + 4 * (n >> 2);
  if constexpr (sizeof(T) == 2)
    gstore_b64(p, __builtin_bit_cast(u32x2, cvt_frag<bf16_t>(x)));
  else
    gstore_b128(p, __builtin_bit_cast(u32x4, x));
}

// Key order of the state tiles of the recurrent kernels.  Row i of a state
// tile set (16 i-rows per accumulator tile) holds key key_of_row(i): within
// each 32-key block, rows 16 h + 4 g + j hold keys 8 g + 4 h + j.  The two
// accumulator tiles of a block then give lane group g the eight consecutive
// keys 8 g .. 8 g + 7 as one 32-deep B operand, and the matching A operand
// (a row of K or Q) is one 16-byte read.  Identity for fewer than 32 keys.
template <int KD>
__host__ __device__ constexpr int key_of_row(int i) {
  return KD < 32 ? i : ((i & ~31) | (((i >> 2) & 3) << 3) | (((i >> 4) & 1) << 2) | (i & 3));
}
template <int KD>
__host__ __device__ constexpr int row_of_key(int k) {
  return KD < 32 ? k : ((k & ~31) | (((k >> 2) & 1) << 4) | (((k >> 3) & 3) << 2) | (k & 3));
}
// First key of the four that lane group g holds in 16-row block kb (the
// others follow consecutively).
template <int KD>
__device__ __forceinline__ int key_col(int kb, int g) { return key_of_row<KD>(16 * kb + 4 * g); }

// The identity as a 16-deep bf16 B fragment: lane (g, n) holds I[4 g + j][n].
__device__ __forceinline__ bf16x4 identity_frag() {
  const int l = lane_id(), g = l >> 4, n = l & 15;
  bf16x4 r;
#pragma unroll
  for (int j = 0; j < 4; ++j) r[j] = (__bf16)((4 * g + j == n) ? 1.f : 0.f);
  return r;
}

// Store a 16 x 16 tile given as a bf16 operand fragment x (lane (g, n) holds
// T[4 g + j][n], the layout of an accumulator converted to bf16) row-major at
// dst (row stride 16).  Fed as the A operand the fragment is T^T, so one
// 16x16x16 MFMA against the identity (id = identity_frag()) leaves T^T I in
// the accumulator layout: lane (g, n) then holds T[n][4 g + j], four
// consecutive elements of row n, written with one 8-byte store.  Every
// product is a bf16 value times one or zero, so the stored values are exact
// copies of the fragment's.  The matrix cores do the lane exchange that would
// otherwise take a dozen VALU instructions per tile.
__device__ __forceinline__ void store_tile16_frag(bf16_t* dst, bf16x4 x, bf16x4 id, int g, int n) {
  f32x4 t = zero4();
  mma16(t, x, id);
  gstore_b64(dst + 16 * n + 4 * g, __builtin_bit_cast(u32x2, cvt_frag<bf16_t>(t)));
}

// ------------------------------------------------ direct global -> LDS copies
// gfx950 loads that write shared memory without a register round trip: every
// active lane l of a wave copies SIZE (4 or 16) bytes from base + off (base
// wave-uniform, off per lane) to LDS bytes [lds + SIZE l, lds + SIZE (l + 1))
// (lds wave-uniform, passed in M0).  They count in vmcnt like other vector
// loads (which complete in issue order for the counter), so a vmcnt wait
// followed by a barrier makes the data visible to the whole workgroup.  They
// are issued from inline assembly: the compiler then neither adds waits for
// them at every barrier nor before unrelated shared-memory reads, and the
// kernels wait for them explicitly with wait_vmcnt.  (A compiler wait for one
// of its own loads stays correct: copies issued after that load only make it
// wait longer.)
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}
// A pointer that the caller knows to be the same in every lane, moved to
// scalar registers (the base of a direct copy must be there; the compiler
// cannot always prove that a pointer built from loaded values is uniform).
template <typename P>
__device__ __forceinline__ P* uniform_ptr(P* p) {
  const uint64_t x = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return (P*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}
// (M0 is written inside the assembly and declared clobbered; the compiler
// warns that it reserves M0, which none of these kernels otherwise use)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
template <int SIZE>
__device__ __forceinline__ void lds_dma(const void* base, uint32_t off, uint32_t lds) {
  static_assert(SIZE == 4 || SIZE == 16, "copy size");
  if constexpr (SIZE == 16)
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(off), "s"(base), "s"(lds) : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
                 :: "v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
#pragma clang diagnostic pop
// Wait until at most N vector memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Wait with a count known only at run time (wave-uniform n; counts above 63
// wait for 63, which is stricter).  A chain of scalar branches selects the
// immediate.
template <int LO, int HI>
__device__ __forceinline__ void wait_vmcnt_rt(int n) {
  if constexpr (LO == HI) {
    wait_vmcnt<LO>();
  } else {
    constexpr int MID = (LO + HI) / 2;
    if (n <= MID)
      wait_vmcnt_rt<LO, MID>(n);
    else
      wait_vmcnt_rt<MID + 1, HI>(n);
  }
}
__device__ __forceinline__ void wait_vmcnt_rt(int n) { wait_vmcnt_rt<0, 63>(n < 63 ? n : 63); }

// Copies issued per wave when the 64-lane blocks of an NB-block copy are
// dealt round-robin to NW waves: the wave with the fewest (the last one).
template <int NB, int NW>
constexpr int dma_min_count() {
  int c = 0;
  for (int i = 0; i * NW + NW - 1 < NB; ++i) ++c;
  return c;
}

// Direct copies of whole tiles and byte ranges into shared memory by a group
// of NW waves: wave w of the group copies the 64-lane blocks w, w + NW, ...
// (1 KiB for tiles).  The *_count functions give the copies each wave issues
// at least (for vmcnt waits: a wave that issues more only waits longer).
template <int NW>
struct GroupDma {
  // The lane index, recomputed at every use: the per-lane offsets of the
  // copies are the same in every chunk step, and hoisted out of a kernel's
  // chunk loop they would hold dozens of registers for its whole length.
  static __device__ __forceinline__ int lane() {
    int x;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(x));
    return x;
  }
  // a coefficient copy uses 16-byte lanes when its 1 KiB blocks split evenly
  // over the waves, else 4-byte lanes when those do
  template <int NBYTES>
  static constexpr int co_size() {
    return (NBYTES % (1024 * NW) == 0) ? 16 : (NBYTES % (256 * NW) == 0) ? 4 : 16;
  }
  template <int NBYTES>
  static constexpr int co_count() {
    constexpr int SZ = co_size<NBYTES>();
    return dma_min_count<(NBYTES + 64 * SZ - 1) / (64 * SZ), NW>();
  }
  template <typename Tile>
  static constexpr int tile_count() {
    return dma_min_count<(Tile::NCHK + 63) / 64, NW>();
  }
  static_assert((NW & (NW - 1)) == 0, "wave groups of 2^n waves");
  // index of the calling wave within its group
  static __device__ __forceinline__ int wid() { return wave_id() & (NW - 1); }

  // Fill a swizzled tile; off(r, c) is the byte offset from the wave-uniform
  // base of logical chunk c of row r.
  template <typename Tile, typename F>
  static __device__ __forceinline__ void tile(Tile& t, const void* base_, F off) {
    constexpr int NB = (Tile::NCHK + 63) / 64;
    const int w = wid(), l = lane();
    const uint32_t lds = lds_addr(t.d);
    const void* base = uniform_ptr(base_);
#pragma unroll
    for (int i = 0; i * NW < NB; ++i) {
      const int blk = i * NW + w;
      if (NB % NW != 0 && blk >= NB) continue;  // wave-uniform
      int r, c;
      Tile::logical(64 * blk + l, r, c);
      if (Tile::NCHK % 64 == 0 || 64 * blk + l < Tile::NCHK)
        lds_dma<16>(base, off(r, c), lds + 1024 * blk);
    }
  }
  // A plain copy of NBYTES contiguous bytes.
  template <int NBYTES>
  static __device__ __forceinline__ void copy(void* dst, const void* src_) {
    constexpr int SZ = co_size<NBYTES>(), NB = (NBYTES + 64 * SZ - 1) / (64 * SZ);
    const int w = wid(), l = lane();
    const uint32_t lds = lds_addr(dst);
    const void* src = uniform_ptr(src_);
#pragma unroll
    for (int i = 0; i * NW < NB; ++i) {
      const int blk = i * NW + w;
      if (NB % NW != 0 && blk >= NB) continue;
      const uint32_t off = 64 * SZ * blk + SZ * l;
      if (NBYTES % (64 * SZ) == 0 || off < (uint32_t)NBYTES)
        lds_dma<SZ>(src, off, lds + 64 * SZ * blk);
    }
  }
  // a tile whose rows are stored row-major, RW elements apart, at src
  template <int RW, typename Tile, typename T>
  static __device__ __forceinline__ void op_tile(Tile& t, const T* src) {
    tile(t, src, [](int r, int c) { return (uint32_t)(sizeof(T) * (r * RW + Tile::EC * c)); });
  }

};

// Unpadded LDS tile of R rows x COLS elements in 16-byte chunks.  Within row
// r the chunk index is XOR-ed with sw(r), so that 16 consecutive rows read at
// the same columns touch 16 distinct chunk positions (fragment reads of a
// 16-row tile are free of bank conflicts) while whole 1 KiB blocks of the
// tile can still be filled by the direct copies above.
template <typename T, int R, int COLS>
struct SwzTile {
  static constexpr int EC = 16 / (int)sizeof(T);  // elements per chunk
  static constexpr int NCH = COLS / EC;           // chunks per row (a power of two)
  static constexpr int NCHK = R * NCH;            // chunks in the tile
  static_assert(COLS % EC == 0 && (NCH & (NCH - 1)) == 0, "rows of 2^n whole chunks");
  alignas(16) T d[R * COLS];
  __device__ static __forceinline__ int sw(int r) {
    return NCH >= 16 ? (r & 15) : ((r * NCH / 16) & (NCH - 1));
  }
  __device__ __forceinline__ const T* at(int r, int col) const {
    return d + r * COLS + ((col / EC) ^ sw(r)) * EC + col % EC;
  }
  // the logical (row, chunk) held at physical chunk position p
  __device__ static __forceinline__ void logical(int p, int& r, int& c) {
    r = p / NCH;
    c = (p % NCH) ^ sw(r);
  }
};

// Rows past T of a row tile (the last, partial chunk): zero them after the
// direct copies have landed.
template <typename Tile>
__device__ __forceinline__ void zero_rows_from(Tile& t, int r0, int nthr) {
  for (int p = threadIdx.x; p < Tile::NCHK; p += nthr)
    if (p / Tile::NCH >= r0) *(uint4*)((char*)t.d + 16 * p) = make_uint4(0, 0, 0, 0);
}

// XCD-aware block mapping: the 8 accelerator dies each have their own L2 and
// receive blocks round-robin by linear id.  Blocks that share a head (the
// value tiles of one head read the same chunk inputs) are placed on one die.
// Returns the (head, tile) pair for a linear block id.
__device__ __forceinline__ void xcd_map(int bid, int nheads, int ntiles, int& head, int& tile) {
  if ((nheads & 7) == 0) {
    const int xcd = bid & 7;
    const int j = bid >> 3;
    tile = j % ntiles;
    head = (j / ntiles) * 8 + xcd;
  } else {
    head = bid / ntiles;
    tile = bid % ntiles;
  }
}

// Row kernels: eight consecutive values of a row held by one lane, as bf16
// (one 16-byte access) or fp32 (two).
template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&x)[8]) {
  if constexpr (sizeof(T) == 2) {
    const uint4 u = *(const uint4*)p;
    const bf16x8 b = __builtin_bit_cast(bf16x8, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = (float)b[i];
  } else {
    const f32x4 a = *(const f32x4*)p, c = *(const f32x4*)(p + 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[i] = a[i];
      x[4 + i] = c[i];
    }
  }
}
template <typename T>
__device__ __forceinline__ void store8(T* p, const float (&x)[8]) {
  if constexpr (sizeof(T) == 2) {
    bf16x8 b;
#pragma unroll
    for (int i = 0; i < 8; ++i) b[i] = (__bf16)x[i];
    *(uint4*)p = __builtin_bit_cast(uint4, b);
  } else {
    *(f32x4*)p = f32x4{x[0], x[1], x[2], x[3]};
    *(f32x4*)(p + 4) = f32x4{x[4], x[5], x[6], x[7]};
  }
}
__device__ __forceinline__ float sigmoidf_(float z) { return 1.f / (1.f + __expf(-z)); }
__device__ __forceinline__ float softplusf_(float y) { return y > 20.f ? y : log1pf(__expf(y)); }

}  // namespace tla
