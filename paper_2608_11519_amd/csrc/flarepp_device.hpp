// Device-side building blocks for the FLARE++ mixer kernels (gfx950, wave64).
//
// All contractions use the 32x32 MFMA tile.  With 64 lanes, lane l belongs to
// half g = l / 32 and column c = l % 32.  For an A operand (32 rows x 16 k)
// lane l holds row c, k = 8g .. 8g+7; for a B operand (16 k x 32 cols) lane l
// holds col c, k = 8g .. 8g+7; the 32x32 fp32 result leaves register r of
// lane l at row 8*(r/4) + 4g + (r%4), column c.  bf16 operands use one
// v_mfma_f32_32x32x16_bf16 per 16-wide k step; fp32 operands use eight
// v_mfma_f32_32x32x2_f32, the j-th taking element j of the same 8-element
// fragment (so both types share one data layout).
#pragma once

#include <hip/hip_runtime.h>
#include <type_traits>
#include <stdint.h>

namespace flarepp {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(8))) float f32x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;

template <typename T> struct Frag;
template <> struct Frag<__bf16> { typedef bf16x8 type; typedef bf16x4 half; };
template <> struct Frag<float> { typedef f32x8 type; typedef f32x4 half; };

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
// Wave index in the block, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }
// A predicate every lane agrees on, made visibly wave-uniform so that the
// compiler emits a scalar branch instead of running both paths under exec.
__device__ __forceinline__ bool uniform(bool p) { return __builtin_amdgcn_readfirstlane((int)p) != 0; }
__device__ __forceinline__ int acc_row(int lane, int r) {
  return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
// Row (within a 16-row group) of element j of half g: the accumulator row
// order of a 32x32 MFMA result, 8 (j / 4) + 4 g + j % 4.
__device__ __forceinline__ int acc_row16(int g, int j) { return 8 * (j >> 2) + 4 * g + (j & 3); }

__device__ __forceinline__ void mma(f32x16& c, const bf16x8& a, const bf16x8& b) {
  c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x16& c, const f32x8& a, const f32x8& b) {
#pragma unroll
  for (int k = 0; k < 8; ++k) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[k], b[k], c, 0, 0, 0);
}

// ---- conversions -----------------------------------------------------------
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ __bf16 from_f32<__bf16>(float x) { return (__bf16)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(__bf16 x) { return (float)x; }

// ---- fragment loads (pointers are aligned to the fragment size) ------------
__device__ __forceinline__ bf16x8 load_frag(const __bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ f32x8 load_frag(const float* p) {
  f32x4 a = *reinterpret_cast<const f32x4*>(p);
  f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
  f32x8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
  r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
  return r;
}
__device__ __forceinline__ bf16x4 load_half(const __bf16* p) {
  return *reinterpret_cast<const bf16x4*>(p);
}
__device__ __forceinline__ f32x4 load_half(const float* p) {
  return *reinterpret_cast<const f32x4*>(p);
}
template <typename T> __device__ __forceinline__ typename Frag<T>::type zero_frag() {
  typename Frag<T>::type z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = from_f32<T>(0.f);
  return z;
}
template <typename T> __device__ __forceinline__ typename Frag<T>::type fill_frag(float v) {
  typename Frag<T>::type z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = from_f32<T>(v);
  return z;
}
template <typename T>
__device__ __forceinline__ typename Frag<T>::type join(typename Frag<T>::half a,
                                                       typename Frag<T>::half b) {
  typename Frag<T>::type r;
#pragma unroll
  for (int i = 0; i < 4; ++i) { r[i] = a[i]; r[4 + i] = b[i]; }
  return r;
}
// Sum of squares of one fragment's elements, in fp32 (bf16: one packed dot
// product per element pair; the squares of bf16 values are exact in fp32).
__device__ __forceinline__ float sumsq(const bf16x8& f) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const bf16x2 v = {f[i], f[i + 1]};
    s = __builtin_amdgcn_fdot2_f32_bf16(v, v, s, false);
  }
  return s;
}
__device__ __forceinline__ float sumsq(const f32x8& f) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s = __builtin_fmaf(f[i], f[i], s);
  return s;
}

// ---- stores of 4 consecutive values ----------------------------------------
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  f32x4 v; v[0] = a; v[1] = b; v[2] = c; v[3] = d;
  *reinterpret_cast<f32x4*>(p) = v;
}
__device__ __forceinline__ void store4(__bf16* p, float a, float b, float c, float d) {
  bf16x4 v; v[0] = (__bf16)a; v[1] = (__bf16)b; v[2] = (__bf16)c; v[3] = (__bf16)d;
  *reinterpret_cast<bf16x4*>(p) = v;
}

// One 32-channel output block of this lane's row in the 32x32 accumulator
// layout (channels 8 q + 4 g .. + 3 hold o[4 q .. 4 q + 3]).  The residual
// is loaded by load_res16 ahead of use, so that a merge issues all its
// residual loads before it waits for any, and store16 adds it (when has_res)
// and stores the block.
template <typename T>
struct Res16 {
  typename Frag<T>::half r[4];
};
template <typename T>
__device__ __forceinline__ void load_res16(Res16<T>& res, const T* rp, int g) {
#pragma unroll
  for (int q = 0; q < 4; ++q) res.r[q] = load_half(rp + 8 * q + 4 * g);
}
template <typename T>
__device__ __forceinline__ void store16(T* op, const f32x16& o, const Res16<T>& res, bool has_res, int g) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float v[4] = {o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]};
    if (has_res) {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += to_f32(res.r[q][e]);
    }
    store4(op + 8 * q + 4 * g, v[0], v[1], v[2], v[3]);
  }
}

// ---- LDS staging ---------------------------------------------------------------
// Wait for every vector memory load of the wave (the copies into LDS among
// them), then a workgroup barrier.
__device__ __forceinline__ void lds_wait_barrier() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
}

// Workgroup barrier over LDS traffic only.  __syncthreads() also waits for
// every global load the wave has in flight (vmcnt counts loads too), which
// would drain a prefetch issued before it; here only this wave's LDS
// operations are waited for.  Use it where the barrier orders LDS accesses
// and nothing written to global memory by another wave is read afterwards.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Copy n16 16-byte chunks src -> LDS dst with direct buffer -> LDS loads by
// all nt threads of the block (each wave fills 1 KiB per step).  The source
// is a raw buffer resource over exactly the n16 chunks (uniform, in scalar
// registers); a step's address is one 32-bit per-thread offset shared by
// every step plus the step's scalar offset, so no per-step 64-bit address
// registers are kept live.
__device__ __forceinline__ void copy_to_lds(const void* src, char* dst, int n16, int nt) {
  if (n16 <= 0) return;
  const int wave = wave_id();
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(src), (short)0, n16 * 16,
                                        0x00020000);  // descriptor word 3: 32-bit data format, raw access
  const int toff = (int)threadIdx.x * 16;
  for (int k = 0; k * nt < n16; ++k) {
    if (k * nt + (int)threadIdx.x < n16)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsrc, (__attribute__((address_space(3))) void*)(dst + (size_t)(k * nt + wave * 64) * 16), 16, toff,
          k * nt * 16, 0, 0);
  }
}

// ---- cross-lane helpers ------------------------------------------------------
// v_permlane32_swap of x with itself: .lo = x of lanes 0..31 in both halves,
// .hi = x of lanes 32..63 in both halves (one VALU instruction, no LDS).
struct HalfPair { float lo, hi; };
__device__ __forceinline__ HalfPair half_pair(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}
// Value held by lane l ^ 32 (the other half of the wave).
__device__ __forceinline__ float other_half(float x) {
  const HalfPair p = half_pair(x);
  return (threadIdx.x & 32) ? p.lo : p.hi;
}
// x of lane l plus x of lane l ^ 32, and their maximum, in every lane.
__device__ __forceinline__ float halves_sum(float x) {
  const HalfPair p = half_pair(x);
  return p.lo + p.hi;
}
__device__ __forceinline__ float halves_max(float x) {
  const HalfPair p = half_pair(x);
  return fmaxf(p.lo, p.hi);
}

// Maximum of a non-negative float over each 32-lane half of the wave, summed
// over the two halves (an upper bound on max_c (x[c] + x[c+32])).  The result
// is wave-uniform.  Non-negative floats order like their bit patterns, so the
// reduction runs on integers through DPP row operations and lane reads.
__device__ __forceinline__ float halfmax_sum_nonneg(float x) {
  int v = __float_as_int(x);
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));  // quad_perm [1,0,3,2]
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));  // quad_perm [2,3,0,1]
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, true)); // row_half_mirror
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, true)); // row_mirror
  int r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
  int r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
  const float s = __int_as_float(max(r0, r1)) + __int_as_float(max(r2, r3));
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(s)));
}

// Maximum of a non-negative float over the whole wave, wave-uniform.
__device__ __forceinline__ float wave_max_nonneg(float x) {
  int v = __float_as_int(x);
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));  // quad_perm [1,0,3,2]
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));  // quad_perm [2,3,0,1]
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, true)); // row_half_mirror
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, true)); // row_mirror
  const int r = max(max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
                    max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
  return __int_as_float(__builtin_amdgcn_readfirstlane(r));
}

// True in every lane when pred holds in every active lane.
__device__ __forceinline__ bool wave_all(bool pred) {
  return __builtin_amdgcn_ballot_w64(!pred) == 0;
}

// ---- one 32-key tile of the routing softmax --------------------------------
// s holds S^T for 32 keys (rows) x 32 queries (cols) in log2 units.  With
// MASK, keys at rows >= nvalid are excluded.  acc is out^T (rows = value
// channels, plus the denominators in row 16 when ONES_ROW); m is the running
// shift per query and ls the denominator partial sums when not ONES_ROW.
//
// tile_shift_free: every score of the tile lies within the shift-free range
// and the shift is 0, so the numerators are bare 2^s.  tile_online: the
// usual online-maximum update.  Kernels run whole loops of one kind (no
// per-tile branch between them), so the accumulators stay in place.
template <bool MASK>
__device__ __forceinline__ void mask_keys(f32x16& s, int nvalid, int lane) {
  if (MASK) {
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (acc_row(lane, e) >= nvalid) s[e] = -INFINITY;
  }
}

template <typename T, int RB, bool ONES_ROW>
__device__ __forceinline__ void pv_product(f32x16 (&acc)[RB], float& ls, const f32x16& s,
                                           const typename Frag<T>::type (&vf)[2][RB]) {
  using F = typename Frag<T>::type;
  constexpr bool BF16 = std::is_same<T, __bf16>::value;
  if (!ONES_ROW && !BF16) {
#pragma unroll
    for (int e = 0; e < 16; ++e) ls += s[e];
  }
  F p0, p1;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    p0[e] = from_f32<T>(s[e]);
    p1[e] = from_f32<T>(s[8 + e]);
  }
  if constexpr (!ONES_ROW && BF16) {
    // the denominators sum the numerators the value product uses (the bf16
    // ones), two per instruction: a dot product of each packed pair with (1, 1)
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 one2 = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      ls = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p0[e], p0[e + 1]}, one2, ls, false);
      ls = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p1[e], p1[e + 1]}, one2, ls, false);
    }
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    mma(acc[rb], vf[0][rb], p0);
    mma(acc[rb], vf[1][rb], p1);
  }
}

template <typename T, int RB, bool ONES_ROW, bool MASK>
__device__ __forceinline__ void tile_shift_free(f32x16 (&acc)[RB], float& ls, f32x16 s,
                                                const typename Frag<T>::type (&vf)[2][RB], int nvalid,
                                                int lane) {
  mask_keys<MASK>(s, nvalid, lane);
#pragma unroll
  for (int e = 0; e < 16; ++e) s[e] = __builtin_amdgcn_exp2f(s[e]);
  pv_product<T, RB, ONES_ROW>(acc, ls, s, vf);
}

template <typename T, int RB, bool ONES_ROW, bool MASK>
__device__ __forceinline__ void tile_online(f32x16 (&acc)[RB], float& m, float& ls, f32x16 s,
                                            const typename Frag<T>::type (&vf)[2][RB], int nvalid, int lane) {
  mask_keys<MASK>(s, nvalid, lane);
  float mx = s[0];
#pragma unroll
  for (int e = 1; e < 16; ++e) mx = fmaxf(mx, s[e]);
  mx = halves_max(mx);
  const float mn = fmaxf(m, mx);
  const float alpha = __builtin_amdgcn_exp2f(m - mn);  // m = -inf -> 0
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[rb][e] *= alpha;
  ls *= alpha;
  m = mn;
#pragma unroll
  for (int e = 0; e < 16; ++e) s[e] = __builtin_amdgcn_exp2f(s[e] - mn);
  pv_product<T, RB, ONES_ROW>(acc, ls, s, vf);
}

// Per-tile choice between the two (used where a loop mixes both kinds).
template <typename T, int RB, bool ONES_ROW>
__device__ __forceinline__ void softmax_pv_tile(f32x16 (&acc)[RB], float& m, float& ls, f32x16 s,
                                                const typename Frag<T>::type (&vf)[2][RB],
                                                int nvalid, bool fast, int lane) {
  if (nvalid < 32) {
    if (fast) {
      m = 0.f;
      tile_shift_free<T, RB, ONES_ROW, true>(acc, ls, s, vf, nvalid, lane);
    } else {
      tile_online<T, RB, ONES_ROW, true>(acc, m, ls, s, vf, nvalid, lane);
    }
  } else if (fast) {
    m = 0.f;
    tile_shift_free<T, RB, ONES_ROW, false>(acc, ls, s, vf, nvalid, lane);
  } else {
    tile_online<T, RB, ONES_ROW, false>(acc, m, ls, s, vf, nvalid, lane);
  }
}

// Softmax denominator of query column c after the last tile: row 16 of the
// value product (ONES_ROW), else the two halves' partial sums.
template <int RB, bool ONES_ROW>
__device__ __forceinline__ float softmax_denominator(const f32x16 (&acc)[RB], float ls, int lane) {
  if (ONES_ROW) return half_pair(acc[0][8]).lo;  // row 16 lives in the lanes of half 0
  return halves_sum(ls);
}

// Upper bound on the squared norm of the rows a fragment set holds (rows are
// split over the two wave halves), wave-uniform.
template <typename T, int NF>
__device__ __forceinline__ float frag_rows_max_sq(const typename Frag<T>::type (&f)[NF]) {
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NF; ++j) s += sumsq(f[j]);
  return halfmax_sum_nonneg(s);
}

}  // namespace flarepp
