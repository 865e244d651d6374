// Backward of the FLARE++ mixer (App. A.5) on gfx950.
//
// * k_gemm: C = sum_seg A B on MFMA 32x32 tiles through LDS, for the
//   projection and W_O gradients (dY = dO W_O^T, dX = sum_j dG_j W_j^T, and
//   in one launch the five weight gradients dW_j = X^T dG_j, dW_O = Y^T dO);
//   the reductions over tokens are split over workgroups (split-K) and summed
//   in a fixed order by k_sum_splits.
// * k_attn_bwd: the SDPA backward of one routing call from its global output
//   and log-normaliser, over a chunk of the long axis (keys of an encode,
//   tokens of the decode).  Each wave owns 32 positions of the long axis and
//   walks the route blocks of a window (operands of the next block in flight
//   in a second register buffer); the long-side gradients stay in registers,
//   the short-side (route) gradients are summed in the wave's LDS slot and,
//   at the end, over the waves in a fixed order into the chunk's partial.
//   Large M x D is covered by several windows, one launch each.
// * k_bwd_reduce sums those partials over the chunks (and over the batch for
//   the shared seeds) in a fixed order; k_bwd_prep lays out the route-side
//   operands of the next call (rows, transposed fragments, c = <dOut, Out>,
//   the log2 normaliser).
// No float atomics anywhere: every result is bitwise reproducible.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "flarepp_device.hpp"
#include "flarepp_internal.hpp"

namespace flarepp {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// ---------------------------------------------------------------------------
// GEMM
// ---------------------------------------------------------------------------
// k step per LDS stage: 64 for bf16, 32 for fp32 (same bytes)
template <typename T> constexpr int gemm_k() { return sizeof(T) == 2 ? 64 : 32; }
// LDS row pitch (elements): the k step plus 16 bytes, so that fragment rows
// start 16-byte aligned and neighbouring rows fall in different banks
template <typename T> constexpr int gemm_pitch() { return gemm_k<T>() + 16 / (int)sizeof(T); }
// LDS offset of element (row i, k) of a staged tile: the 8-element blocks of
// a row are permuted by the row's group of 8 (block ^ (i / 8)), so that the
// k-pair stores of eight rows 8 apart fall in different banks; a fragment
// (8 consecutive k from a multiple of 8) stays contiguous.
template <typename T>
__device__ __forceinline__ int gemm_lds(int i, int k) {
  constexpr int NB = gemm_k<T>() / 8;
  return i * gemm_pitch<T>() + ((((k >> 3) ^ (i >> 3)) & (NB - 1)) << 3) + (k & 7);
}

__device__ __forceinline__ void load8(const __bf16* p, float (&v)[8]) {
  const bf16x8 x = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = (float)x[j];
}
__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int j = 0; j < 4; ++j) { v[j] = a[j]; v[4 + j] = b[j]; }
}
__device__ __forceinline__ void store8(__bf16* p, const float (&v)[8]) {
  bf16x8 x;
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = (__bf16)v[j];
  *reinterpret_cast<bf16x8*>(p) = x;
}
__device__ __forceinline__ void store8(float* p, const float (&v)[8]) {
  f32x4 a, b;
#pragma unroll
  for (int j = 0; j < 4; ++j) { a[j] = v[j]; b[j] = v[4 + j]; }
  *reinterpret_cast<f32x4*>(p) = a;
  *reinterpret_cast<f32x4*>(p + 4) = b;
}
__device__ __forceinline__ void store_pair(__bf16* p, float a, float b) {
  bf16x2_t v;
  v[0] = (__bf16)a; v[1] = (__bf16)b;
  *reinterpret_cast<bf16x2_t*>(p) = v;
}
__device__ __forceinline__ void store_pair(float* p, float a, float b) {
  f32x2 v;
  v[0] = a; v[1] = b;
  *reinterpret_cast<f32x2*>(p) = v;
}

// Element j of fragments a and b (k and k + 1 of one row) as one k pair.
// bf16: the two 16-bit halves are picked by a byte permute, no conversion.
__device__ __forceinline__ void store_kpair(__bf16* p, const bf16x8& a, const bf16x8& b, int j) {
  typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
  const u32x4 ua = __builtin_bit_cast(u32x4, a), ub = __builtin_bit_cast(u32x4, b);
  // result bytes {a.lo, b.lo} for even j, {a.hi, b.hi} for odd j
  *reinterpret_cast<unsigned int*>(p) =
      __builtin_amdgcn_perm(ub[j >> 1], ua[j >> 1], (j & 1) ? 0x07060302u : 0x05040100u);
}
__device__ __forceinline__ void store_kpair(float* p, const f32x8& a, const f32x8& b, int j) {
  store_pair(p, a[j], b[j]);
}

// One ROWS x K operand tile, staged through registers into LDS as rows of k:
// row i, column k holds X(row0 + i, k0 + k) where X(i, k) = x[i * s_i + k *
// s_k].  Unit stride along k: runs of 8 k values (16-byte loads and stores).
// Otherwise (unit stride along i): runs of 8 rows for two neighbouring k,
// stored as k pairs.  The host keeps unit-stride runs 8-element aligned.
// gemm_load issues the global loads of a tile; gemm_store writes them to LDS
// later, so the loads of the next k step overlap the current one's MFMAs.
template <typename T, int ROWS>
struct GemmStage {
  static constexpr int K = gemm_k<T>();
  static constexpr int NK = (ROWS * (K / 8) + 255) / 256;      // k runs per thread
  static constexpr int NP = ((ROWS / 8) * (K / 2) + 255) / 256;  // row-run pairs per thread
  static constexpr int NF = NK > 2 * NP ? NK : 2 * NP;
  typename Frag<T>::type f[NF];
};

// 16-byte aligned stores of a fragment (fp32: two 16-byte halves)
__device__ __forceinline__ void store_frag8(__bf16* p, const bf16x8& f) { *reinterpret_cast<bf16x8*>(p) = f; }
__device__ __forceinline__ void store_frag8(float* p, const f32x8& f) {
  f32x4 a, b;
#pragma unroll
  for (int j = 0; j < 4; ++j) { a[j] = f[j]; b[j] = f[4 + j]; }
  *reinterpret_cast<f32x4*>(p) = a;
  *reinterpret_cast<f32x4*>(p + 4) = b;
}

template <typename T>
__device__ __forceinline__ typename Frag<T>::type frag_from(const float (&v)[8]) {
  typename Frag<T>::type f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = from_f32<T>(v[j]);
  return f;
}

template <typename T, int ROWS>
__device__ __forceinline__ void gemm_load(GemmStage<T, ROWS>& st, const T* x, int64_t s_i, int64_t s_k, int row0,
                                          int nrows, int k0, int kend) {
  constexpr int K = gemm_k<T>();
  const int t = threadIdx.x;
  if (s_k == 1) {
    constexpr int RPR = K / 8;  // runs per row
#pragma unroll
    for (int q = 0; q < GemmStage<T, ROWS>::NK; ++q) {
      const int r = t + 256 * q;
      if (r >= ROWS * RPR) break;
      const int ii = r / RPR, kk = (r % RPR) * 8;
      const int i = row0 + ii, k = k0 + kk;
      if (i < nrows && k + 8 <= kend) {
        st.f[q] = load_frag(x + (int64_t)i * s_i + k);
      } else {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (i < nrows && k + j < kend) ? to_f32(x[(int64_t)i * s_i + k + j]) : 0.f;
        st.f[q] = frag_from<T>(v);
      }
    }
  } else {
    constexpr int IG = ROWS / 8;  // groups of 8 rows
#pragma unroll
    for (int q = 0; q < GemmStage<T, ROWS>::NP; ++q) {
      const int r = t + 256 * q;
      if (r >= IG * (K / 2)) break;
      const int ii = (r % IG) * 8, kk = 2 * (r / IG);
      const int i = row0 + ii, k = k0 + kk;
      if (s_i == 1 && i + 8 <= nrows && k + 2 <= kend) {
        st.f[2 * q] = load_frag(x + (int64_t)k * s_k + i);
        st.f[2 * q + 1] = load_frag(x + (int64_t)(k + 1) * s_k + i);
      } else {
        float v[8], w[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          v[j] = (i + j < nrows && k < kend) ? to_f32(x[(int64_t)(i + j) * s_i + (int64_t)k * s_k]) : 0.f;
          w[j] = (i + j < nrows && k + 1 < kend) ? to_f32(x[(int64_t)(i + j) * s_i + (int64_t)(k + 1) * s_k]) : 0.f;
        }
        st.f[2 * q] = frag_from<T>(v);
        st.f[2 * q + 1] = frag_from<T>(w);
      }
    }
  }
}

template <typename T, int ROWS>
__device__ __forceinline__ void gemm_store(const GemmStage<T, ROWS>& st, T* dst, int64_t s_k) {
  constexpr int K = gemm_k<T>();
  const int t = threadIdx.x;
  if (s_k == 1) {
    constexpr int RPR = K / 8;
#pragma unroll
    for (int q = 0; q < GemmStage<T, ROWS>::NK; ++q) {
      const int r = t + 256 * q;
      if (r >= ROWS * RPR) break;
      store_frag8(dst + gemm_lds<T>(r / RPR, (r % RPR) * 8), st.f[q]);
    }
  } else {
    constexpr int IG = ROWS / 8;
#pragma unroll
    for (int q = 0; q < GemmStage<T, ROWS>::NP; ++q) {
      const int r = t + 256 * q;
      if (r >= IG * (K / 2)) break;
      const int ii = (r % IG) * 8, kk = 2 * (r / IG);
#pragma unroll
      for (int j = 0; j < 8; ++j) store_kpair(dst + gemm_lds<T>(ii + j, kk), st.f[2 * q], st.f[2 * q + 1], j);
    }
  }
}

// Workgroup tile TM x TN (64 or 128 each), four waves in a 2 x 2 grid, each
// wave (TM / 64) x (TN / 64) accumulators of 32 x 32.  The global loads of
// k step s + 1 are in flight while step s runs on the MFMAs.
template <typename T, int TM, int TN>
__global__ __launch_bounds__(256) void k_gemm(GemmParams p) {
  constexpr int K = gemm_k<T>(), PITCH = gemm_pitch<T>(), MT = TM / 64, NT = TN / 64;
  static_assert(gemm_k<T>() % 16 == 0, "k step");
  __shared__ __attribute__((aligned(16))) T As[TM * PITCH];
  __shared__ __attribute__((aligned(16))) T Bs[TN * PITCH];
  const int lane = lane_id(), wave = wave_id(), g = lane >> 5, c = lane & 31;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;
  int prob = blockIdx.z / p.splits, z = blockIdx.z % p.splits;
  if (p.nprob > 1 && gridDim.x * gridDim.y == 1) {
    // one output tile per problem (C <= 128): the problems of one token
    // chunk go to the same XCD (workgroups are dealt to the 8 XCDs in turn),
    // close together in time, so the X rows they share come from that
    // XCD's L2 after the first read; z runs over the chunks rounded up to 8
    const int L = blockIdx.z, xcd = L & 7, r = L >> 3;
    prob = r % p.nprob;
    z = (r / p.nprob) * 8 + xcd;
    if (z >= p.splits) return;  // whole workgroup, before any barrier
  }
  const int kbeg = z * p.kchunk, kend = min(p.K, kbeg + p.kchunk);
  const int mw = wave >> 1, nw = wave & 1;
  f32x16 acc[MT][NT];
#pragma unroll
  for (int a = 0; a < MT; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;
  // this problem's segments; a null b operand ends the list early
  const int seg0 = prob * p.nseg;
  int seg1 = seg0 + 1;
  while (seg1 < seg0 + p.nseg && p.b[seg1]) ++seg1;
  // the (segment, k step) sequence of this workgroup, walked with a one-step
  // register prefetch
  const int nk = kend > kbeg ? (kend - kbeg + K - 1) / K : 0;
  const int nsteps = (seg1 - seg0) * nk;
  GemmStage<T, TM> sa;
  GemmStage<T, TN> sb;
  auto load_step = [&](int it) __attribute__((always_inline)) {
    const int seg = seg0 + it / nk, k0 = kbeg + (it % nk) * K;
    gemm_load(sa, static_cast<const T*>(p.a[seg]), p.a_m, p.a_k, m0, p.M, k0, kend);
    gemm_load(sb, static_cast<const T*>(p.b[seg]), p.b_n, p.b_k, n0, p.N, k0, kend);
  };
  if (nsteps > 0) load_step(0);
  for (int it = 0; it < nsteps; ++it) {
    gemm_store(sa, As, p.a_k);
    gemm_store(sb, Bs, p.b_k);
    __syncthreads();
    if (it + 1 < nsteps) load_step(it + 1);
#pragma unroll
    for (int ks = 0; ks < K / 16; ++ks) {
      typename Frag<T>::type af[MT], bfr[NT];
#pragma unroll
      for (int a = 0; a < MT; ++a) af[a] = load_frag(As + gemm_lds<T>(32 * (MT * mw + a) + c, 16 * ks + 8 * g));
#pragma unroll
      for (int b = 0; b < NT; ++b) bfr[b] = load_frag(Bs + gemm_lds<T>(32 * (NT * nw + b) + c, 16 * ks + 8 * g));
      // C^T = B^T A^T: the accumulator's rows are output columns, so each
      // lane holds runs of 4 consecutive columns of one output row
#pragma unroll
      for (int a = 0; a < MT; ++a)
#pragma unroll
        for (int b = 0; b < NT; ++b) mma(acc[a][b], bfr[b], af[a]);
    }
    __syncthreads();
  }
  const int64_t base = ((int64_t)prob * p.splits + z) * p.split_stride;
#pragma unroll
  for (int a = 0; a < MT; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b) {
      const int m = m0 + 32 * (MT * mw + a) + c;
      if (m >= p.M) continue;
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int n = n0 + 32 * (NT * nw + b) + acc_row(lane, 4 * r4);  // 4 columns n .. n + 3
        const int64_t o = base + (int64_t)m * p.ldc + n;
        const float v[4] = {acc[a][b][4 * r4], acc[a][b][4 * r4 + 1], acc[a][b][4 * r4 + 2], acc[a][b][4 * r4 + 3]};
        if (n + 3 < p.N) {
          if (p.c_t) store4(static_cast<T*>(p.c) + o, v[0], v[1], v[2], v[3]);
          else store4(static_cast<float*>(p.c) + o, v[0], v[1], v[2], v[3]);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (n + q < p.N) {
              if (p.c_t) static_cast<T*>(p.c)[o + q] = from_f32<T>(v[q]);
              else static_cast<float*>(p.c)[o + q] = v[q];
            }
        }
      }
    }
}

// s + x[0] + x[st] + ... + x[(n - 1) st], added in that order; the loads of
// a group of 8 are issued before its adds.
__device__ __forceinline__ float sum_run(float s, const float* x, int64_t st, int n) {
  int r = 0;
  for (; r + 8 <= n; r += 8) {
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = x[(int64_t)(r + j) * st];
#pragma unroll
    for (int j = 0; j < 8; ++j) s += v[j];
  }
  for (; r < n; ++r) s += x[(int64_t)r * st];
  return s;
}

struct SumOuts {
  float* out[5];
};

__global__ __launch_bounds__(256) void k_sum_splits(const float* part, SumOuts o, int64_t n, int splits, int nprob) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n * nprob) return;
  const int pr = (int)(i / n);
  const int64_t e = i % n;
  o.out[pr][e] = sum_run(0.f, part + (int64_t)pr * splits * n + e, n, splits);
}

// ---------------------------------------------------------------------------
// SDPA backward over a chunk of the long axis
// ---------------------------------------------------------------------------
// LDS per wave: the short-side slot(s) [D][Mp + 4] fp32 (route index fastest,
// padded so that the lanes' rows fall in different banks) and one transpose
// tile [32][32 + 16 bytes] of T (dS, then P in the decode); per workgroup
// (encode) the routes' L and c.
template <typename T> constexpr int tb_pitch() { return 32 + 16 / (int)sizeof(T); }
// Bytes of a wave's tile buffer: the transpose tile, or for the bf16 decode
// at D = 16 its staged long-side rows (keys, dY, Y: 1 KiB each, then 32
// log-normalisers), whichever is larger.
constexpr size_t attn_bwd_tile_bytes(int D, bool dec, int elem_bytes) {
  const size_t tile = (size_t)32 * (32 + 16 / elem_bytes) * elem_bytes;
  const size_t staged = (dec && elem_bytes == 2 && D == 16) ? 3 * 1024 + 128 : 0;
  return tile > staged ? tile : staged;
}
size_t attn_bwd_wave_bytes(int D, int nsb, bool dec, int elem_bytes) {
  return sizeof(float) * (size_t)(dec ? 2 : 1) * D * (32 * nsb + 4) + attn_bwd_tile_bytes(D, dec, elem_bytes);
}

// Fragment of a long-side row: element j = x[n * sn + (d0 + j) * sd] (one
// 16-byte load when the row is contiguous), zero when !ok.  The caller passes
// an in-range row n even when !ok, so the loads need no branch.
template <typename T>
__device__ __forceinline__ typename Frag<T>::type long_frag(const T* x, int64_t sn, int64_t sd, int n, int d0, bool ok) {
  typename Frag<T>::type f;
  if (sd == 1) {
    f = load_frag(x + (int64_t)n * sn + d0);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = x[(int64_t)n * sn + (int64_t)(d0 + j) * sd];
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = ok ? f[j] : from_f32<T>(0.f);
  return f;
}

// Route-side operands of one block of 32 routes, loaded one block ahead.
// Store 4 long-side values at out[o], adding what is there when acc.  With a
// lo buffer the value is kept as hi = T(v) in out and lo = T(v - hi) in lo:
// about 16 mantissa bits in bf16, so the token reductions over it (the weight
// gradients) do not lose the small token-dependent part of a gradient whose
// tokens share a large common part.
template <typename T>
__device__ __forceinline__ void long_store(T* out, T* lo, int64_t o, int acc, float (&v)[4]) {
  if (acc) {
    const typename Frag<T>::half old = load_half(out + o);
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] += to_f32(old[q]);
    if (lo) {
      const typename Frag<T>::half ol = load_half(lo + o);
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] += to_f32(ol[q]);
    }
  }
  store4(out + o, v[0], v[1], v[2], v[3]);
  if (lo) {
    float r[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = v[q] - to_f32(from_f32<T>(v[q]));
    store4(lo + o, r[0], r[1], r[2], r[3]);
  }
}

template <typename T, int D, bool DEC>
struct ShortBlock {
  static constexpr int KS = D / 16, DB = (D + 31) / 32;
  typename Frag<T>::type a[KS], gr[KS];       // rows of A_sh and G_sh
  typename Frag<T>::type at[2][DB], gt[2][DB];  // transposed fragments (gt: encode)
};

template <typename T, int D, bool DEC>
__device__ __forceinline__ void load_short(ShortBlock<T, D, DEC>& s, const T* ash, const T* gsh, const T* asht,
                                           const T* gsht, int sb, int lane) {
  constexpr int KS = D / 16, DB = (D + 31) / 32;
  const int g = lane >> 5, c = lane & 31;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    s.a[ks] = load_frag(ash + (32 * sb + c) * D + 16 * ks + 8 * g);
    s.gr[ks] = load_frag(gsh + (32 * sb + c) * D + 16 * ks + 8 * g);
  }
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int fo = (((sb * 2 + kk) * DB + db) * 64 + lane) * 8;
      s.at[kk][db] = load_frag(asht + fo);
      if constexpr (!DEC) s.gt[kk][db] = load_frag(gsht + fo);
    }
}

// bf16 at D = 16 keeps two waves per SIMD (two workgroups per CU)
template <typename T, int D, bool DEC>
__global__ __launch_bounds__(256, (sizeof(T) == 2 && D == 16) ? 2 : 1) void k_attn_bwd(AttnBwdParams p) {
  using F = typename Frag<T>::type;
  constexpr int KS = D / 16, DB = (D + 31) / 32, TBP = tb_pitch<T>();
  constexpr int TBE = (int)(attn_bwd_tile_bytes(D, DEC, (int)sizeof(T)) / sizeof(T));  // tile buffer elements
  // bf16: dS (and P in the decode) change layout on the MFMA (times a
  // permutation matrix) instead of through LDS; fp32 keeps the LDS transpose
  constexpr bool MT = std::is_same<T, __bf16>::value;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int lane = lane_id(), g = lane >> 5, c = lane & 31, wave = wave_id();
  // position of element j of the lane's k = position fragment kk in the
  // short-side products: 16 kk + 8 g + j with the LDS transpose; with the
  // MFMA one it is the accumulator's row order, 16 kk + 8 (j / 4) + 4 g + j % 4
  auto short_k_pos = [&](int kk, int gg, int j) __attribute__((always_inline)) {
    return MT ? 16 * kk + 8 * (j >> 2) + 4 * gg + (j & 3) : 16 * kk + 8 * gg + j;
  };
  // B operands of the layout change: perm[kk][k = 8 g + j][col = c] = 1 when
  // route 16 kk + 8 (j / 4) + 4 g + j % 4 (the route that the accumulator's
  // element 8 kk + j of lane (., g) holds) is c
  F perm[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int j = 0; j < 8; ++j) perm[kk][j] = from_f32<T>(short_k_pos(kk, g, j) == c ? 1.f : 0.f);
  const int W = blockDim.x >> 6;
  const int bh = blockIdx.x / p.R, r = blockIdx.x % p.R;
  const int b = bh / p.H, h = bh % p.H;
  const int SB0 = p.sb0, NS = p.nsb, SP = 32 * NS + 4;  // this launch's route blocks
  const int slot_floats = (DEC ? 2 : 1) * D * SP;
  float* slot_a = reinterpret_cast<float*>(smem) + wave * slot_floats;
  float* slot_g = slot_a + D * SP;
  T* tb = reinterpret_cast<T*>(reinterpret_cast<float*>(smem) + W * slot_floats) + wave * TBE;
  // encode: the routes' -L (log2) and -c of this (b, h), [2][Mp], after the
  // waves' transpose tiles (the initial values of the S and dP accumulators)
  float* lc_lds = reinterpret_cast<float*>(reinterpret_cast<T*>(reinterpret_cast<float*>(smem) + W * slot_floats) +
                                           W * TBE);
  for (int i = lane; i < slot_floats; i += 64) slot_a[i] = 0.f;
  if constexpr (!DEC) {
    for (int i = threadIdx.x; i < 2 * p.Mp; i += blockDim.x)
      lc_lds[i] = -(i < p.Mp ? p.lrow[(int64_t)bh * p.Mp + i] : p.crow[(int64_t)bh * p.Mp + i - p.Mp]);
    __syncthreads();
  }

  const T* ash = static_cast<const T*>(p.ash) + b * p.ash_sb + h * p.ash_sh;
  const T* asht = static_cast<const T*>(p.asht) + b * p.asht_sb + h * p.asht_sh;
  const T* gsh = static_cast<const T*>(p.gsh) + b * p.gsh_sb + h * p.gsh_sh;
  const T* gsht = DEC ? nullptr : static_cast<const T*>(p.gsht) + b * p.gsht_sb + h * p.gsht_sh;
  const T* blo = static_cast<const T*>(p.blo) + b * p.blo_sb + h * p.blo_sh;
  const T* glo = static_cast<const T*>(p.glo) + b * p.glo_sb + h * p.glo_sh;
  T* dout_b = static_cast<T*>(p.dout_b);
  T* dout_g = static_cast<T*>(p.dout_g);

  // bf16 at D = 16 with token-major keys: a tile's long-side rows are copied
  // into the wave's tile buffer one tile ahead by direct buffer -> LDS loads,
  // issued as soon as the current tile's rows have been read out, so no tile
  // waits on its loads.  Encode: the 32 key rows [32][16], then the 16 d-major
  // value rows of its 32 positions [16][32]; decode: key rows, dY rows, Y rows
  // ([32][16] each), then the 32 log-normalisers; 1 KiB per block of rows.
  // Rows past the long length read as zero (buffer bounds; the d-major
  // values are zero-padded).
  constexpr bool STG = MT && D == 16;
  const bool stg = STG && p.blo_sd == 1 && p.blo_sn == D &&
                   (DEC ? (p.glo_sd == 1 && p.ylo_sn == p.glo_sn) : p.glo_sn == 1);  // uniform
  const T* ylo = DEC ? static_cast<const T*>(p.ylo) + b * p.ylo_sb + h * p.ylo_sh : nullptr;
  auto stage_issue = [&](int i) __attribute__((always_inline)) {
    if (i >= p.tpw) return;
    const int n0i = ((r * p.tpw + i) * W + wave) * 32;  // wave-uniform
    if (n0i >= p.Nl) return;
    constexpr int EB = (int)sizeof(T);
    const int kbytes = (int)std::min<int64_t>((int64_t)p.Nl * D * EB, 0x7fffffff);
    const int vbytes = (int)std::min<int64_t>((int64_t)D * p.glo_sd * EB, 0x7fffffff);
    const __amdgpu_buffer_rsrc_t rk =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(blo), (short)0, kbytes, 0x00020000);
    // lane l: key row n0i + l / 2, half l % 2 (likewise dY and Y rows);
    // value row l / 4, positions n0i + 8 (l % 4) .. + 7; each lands at byte
    // 16 l of its KiB
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (__attribute__((address_space(3))) void*)tb, 16,
                                             (n0i * D + 8 * lane) * EB, 0, 0, 0);
    if constexpr (DEC) {
      const int sn = (int)p.glo_sn;
      const int rbytes = (int)std::min<int64_t>((int64_t)p.Nl * sn * EB, 0x7fffffff);
      const __amdgpu_buffer_rsrc_t rg =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(glo), (short)0, rbytes, 0x00020000);
      const __amdgpu_buffer_rsrc_t ry =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(ylo), (short)0, rbytes, 0x00020000);
      const int roff = ((n0i + (lane >> 1)) * sn + 8 * (lane & 1)) * EB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rg, (__attribute__((address_space(3))) void*)(tb + 32 * D), 16, roff, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, (__attribute__((address_space(3))) void*)(tb + 64 * D), 16, roff, 0, 0, 0);
      if (lane < 8) {  // 32 log-normalisers, 4 per lane
        const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float*>(p.lcol + (int64_t)bh * p.Nl), (short)0,
            (int)std::min<int64_t>((int64_t)p.Nl * 4, 0x7fffffff), 0x00020000);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (__attribute__((address_space(3))) void*)(tb + 96 * D), 16,
                                                 (n0i + 4 * lane) * 4, 0, 0, 0);
      }
    } else {
      const __amdgpu_buffer_rsrc_t rv =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(glo), (short)0, vbytes, 0x00020000);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (__attribute__((address_space(3))) void*)(tb + 32 * D), 16,
                                               ((lane >> 2) * (int)p.glo_sd + n0i + 8 * (lane & 3)) * EB, 0, 0, 0);
    }
    asm volatile("" ::: "memory");  // the copies go out ahead of the tile's route-operand loads
  };
  if (stg) {
    // zero the tile buffer first: rows past the long length hold zeros (or,
    // after a full tile, that tile's finite rows) whatever the bounds-checked
    // copies leave there, so no NaN of earlier LDS contents reaches a sum
    for (int i = 8 * lane; i < TBE; i += 8 * 64) store_frag8(tb + i, zero_frag<T>());
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    stage_issue(0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  for (int i = 0; i < p.tpw; ++i) {
    const int n0 = ((r * p.tpw + i) * W + wave) * 32;  // wave-uniform
    if (n0 >= p.Nl) break;
    const int n = n0 + c;
    const bool nok = n < p.Nl;
    const int nc = nok ? n : p.Nl - 1;        // in-range row for the loads
    const bool full_tile = n0 + 32 <= p.Nl;  // wave-uniform: no position masked
    // long-side B operands of S (keys) and dP (values), one lane per position
    F kb[KS], gb[KS];
    // long-side B operands of the short-side products (k = position, n = d)
    F kt[2][DB], gt[2][DB];
    // decode: c = <dY_n, Y_n> and the token's log-normaliser
    float Ll = 0.f, cl = 0.f;
    if (stg) {
      // from the staged rows (landed at the end of the previous tile)
      // (the lane index is re-read here so that the per-lane LDS offsets are
      // computed per tile rather than held in registers across the loop)
      int ln = lane;
      asm volatile("" : "+v"(ln));
      const int lg = ln >> 5, lc = ln & 31;
      const T* sk = tb;           // [32 positions][D]
      const T* sv = tb + 32 * D;  // encode: [D][32 positions]; decode: dY [32 positions][D]
      kb[0] = load_frag(sk + lc * D + 8 * lg);
      // columns d = lc >= D of the short-side products are never stored:
      // those lanes read a valid (finite) value of another column
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int j = 0; j < 8; ++j) kt[kk][0][j] = sk[short_k_pos(kk, lg, j) * D + (lc & (D - 1))];
      if constexpr (DEC) {
        gb[0] = load_frag(sv + lc * D + 8 * lg);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int j = 0; j < 8; ++j) gt[kk][0][j] = sv[short_k_pos(kk, lg, j) * D + (lc & (D - 1))];
        // c = <dY_n, Y_n> over the head's channels and the token's
        // log-normaliser (log2 units), from the staged rows
        const F yf = load_frag(tb + 64 * D + lc * D + 8 * lg);
        float sacc = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) sacc += to_f32(gb[0][j]) * to_f32(yf[j]);
        cl = sacc + other_half(sacc);
        Ll = reinterpret_cast<const float*>(tb + 96 * D)[lc];
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) gb[0][j] = sv[(8 * lg + j) * 32 + lc];
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // read out before the next tile's rows land
      stage_issue(i + 1);
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kb[ks] = long_frag(blo, p.blo_sn, p.blo_sd, nc, 16 * ks + 8 * g, nok);
      if (D == 32 && p.glo_sn == 1) {  // wave-uniform (at D = 16 the staging would cost the second wave per SIMD)
        // d-major values (each head's rows padded to whole 32-position tiles):
        // the tile's D rows of 32 positions go through the wave's transpose
        // tile with 16-byte loads (chunk r: row r / 4, positions 8 (r % 4) ..
        // + 7), then each lane reads its position's column
#pragma unroll
        for (int r0 = 0; r0 < D * 4; r0 += 64) {
          const int r = r0 + lane, d = r >> 2, q = r & 3;
          store_frag8(tb + d * TBP + 8 * q, load_frag(glo + (int64_t)d * p.glo_sd + n0 + 8 * q));
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const T v = tb[(16 * ks + 8 * g + j) * TBP + c];
            gb[ks][j] = nok ? v : from_f32<T>(0.f);
          }
        __builtin_amdgcn_wave_barrier();
      } else {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) gb[ks] = long_frag(glo, p.glo_sn, p.glo_sd, nc, 16 * ks + 8 * g, nok);
      }
      // row-major long side (unit stride along d): each lane stores its
      // position's row of 32 columns into the wave's transpose tile with
      // 16-byte loads, then reads one column (d = 32 db + c) of it
      auto transpose_long = [&](const T* x, int64_t sn, F (&out)[2][DB]) __attribute__((always_inline)) {
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int d0 = 32 * db + 16 * g + 8 * h;  // D is a multiple of 16: d0 < D means d0 + 8 <= D
            store_frag8(tb + c * TBP + 16 * g + 8 * h, d0 < D ? load_frag(x + (int64_t)nc * sn + d0) : zero_frag<T>());
          }
          __builtin_amdgcn_wave_barrier();
#pragma unroll
          for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const int pos = short_k_pos(kk, g, j);
              const T v = tb[pos * TBP + c];
              out[kk][db][j] = n0 + pos < p.Nl ? v : from_f32<T>(0.f);
            }
          __builtin_amdgcn_wave_barrier();
        }
      };
      // (D = 64 keeps the element loads: the staged rows would add to a
      // register budget that is already full there)
      if (D <= 32 && p.blo_sd == 1 && (!DEC || p.glo_sd == 1)) {  // wave-uniform
        transpose_long(blo, p.blo_sn, kt);
        if constexpr (DEC) transpose_long(glo, p.glo_sn, gt);
      } else {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const int nn = n0 + short_k_pos(kk, g, j), d = 32 * db + c;
              const bool ok = nn < p.Nl && d < D;
              const int64_t at = (int64_t)min(nn, p.Nl - 1) * p.blo_sn + (int64_t)min(d, D - 1) * p.blo_sd;
              const T kv = blo[at];
              kt[kk][db][j] = ok ? kv : from_f32<T>(0.f);
              if (DEC) {
                const T gv = glo[(int64_t)min(nn, p.Nl - 1) * p.glo_sn + (int64_t)min(d, D - 1) * p.glo_sd];
                gt[kk][db][j] = ok ? gv : from_f32<T>(0.f);
              }
            }
      }
    }
    // decode: c = <dY_n, Y_n> over the head's channels, and the token's
    // log-normaliser over the routes (log2 units) from the forward
    if (DEC && !stg) {
      const T* y = ylo;
      float sacc = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const F yf = long_frag(y, p.ylo_sn, (int64_t)1, nc, 16 * ks + 8 * g, nok);
#pragma unroll
        for (int j = 0; j < 8; ++j) sacc += to_f32(gb[ks][j]) * to_f32(yf[j]);
      }
      cl = sacc + other_half(sacc);
      Ll = p.lcol[(int64_t)bh * p.Nl + nc];
    }

    f32x16 dk[DB], dv[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) dk[db][e] = dv[db][e] = 0.f;
    // initial accumulators of route block sb: encode -L and -c of the block's
    // routes (rows), so that S' = s log2(e) S - L and dP' = dP - c come out
    // of the MFMAs; decode zero (L and c belong to the column there).  The
    // ash rows are scaled by s log2(e) beforehand.
    auto load_init = [&](int sb, f32x16& si, f32x16& di) __attribute__((always_inline)) {
      if constexpr (!DEC) {
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(lc_lds + 32 * (SB0 + sb) + 8 * a + 4 * g);
          const f32x4 c4 = *reinterpret_cast<const f32x4*>(lc_lds + p.Mp + 32 * (SB0 + sb) + 8 * a + 4 * g);
#pragma unroll
          for (int q = 0; q < 4; ++q) { si[4 * a + q] = l4[q]; di[4 * a + q] = c4[q]; }
        }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) si[e] = di[e] = 0.f;
      }
    };
    // one block of 32 routes; the operands of the next block are loaded into
    // the other buffer first (the last block again at the end, so the same
    // number of loads is in flight on every block), and its initial
    // accumulators at the end
    auto route_block = [&](const ShortBlock<T, D, DEC>& cb, int sb, f32x16& si, f32x16& di) __attribute__((always_inline)) {
      f32x16 sc = si, dp = di;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        mma(sc, cb.a[ks], kb[ks]);
        mma(dp, cb.gr[ks], gb[ks]);
      }
      // P = exp2(S'), dS = P dP' (encode; decode: the column's L and c
      // subtracted here); rows past M and columns past the long length are
      // zero
      f32x16 P, dS;
      auto softmax_grad = [&](auto masked) __attribute__((always_inline)) {
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          float pv, dd;
          if constexpr (DEC) {
            pv = __builtin_amdgcn_exp2f(sc[rr] - Ll);
            dd = dp[rr] - cl;
          } else {
            pv = __builtin_amdgcn_exp2f(sc[rr]);
            dd = dp[rr];
          }
          if constexpr (decltype(masked)::value)
            if (!(nok && 32 * (SB0 + sb) + acc_row(lane, rr) < p.M)) pv = 0.f;
          P[rr] = pv;
          dS[rr] = pv * dd;
        }
      };
      if (full_tile && 32 * (SB0 + sb + 1) <= p.M) softmax_grad(std::false_type{});  // wave-uniform
      else softmax_grad(std::true_type{});
      // P and dS as B operands (k = route, in the accumulator's row order)
      F pb[2], dsb[2];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          pb[kk][j] = from_f32<T>(P[8 * kk + j]);
          dsb[kk][j] = from_f32<T>(dS[8 * kk + j]);
        }
      // long side: dB^T += A^T dS, dG^T += G^T P (encode)
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          mma(dk[db], cb.at[kk][db], dsb[kk]);
          if constexpr (!DEC) mma(dv[db], cb.gt[kk][db], pb[kk]);
        }
      // short side: dS (then P in the decode) with rows = routes along the
      // lanes and k = positions in the registers
      F dsa[2], pa[2];
      if constexpr (MT) {
        // (dS^T)^T on the MFMA: A = dS^T (rows = positions, k = routes in the
        // accumulator's order, exactly the B operand dsb already built) times
        // the permutation perm gives dS with lane = route and the positions
        // in the accumulator's row order; exact (one product of 1 per sum)
        auto relayout = [&](const F (&src)[2], F (&dst)[2]) __attribute__((always_inline)) {
          f32x16 t;
#pragma unroll
          for (int e = 0; e < 16; ++e) t[e] = 0.f;
          mma(t, src[0], perm[0]);
          mma(t, src[1], perm[1]);
#pragma unroll
          for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int j = 0; j < 8; ++j) dst[kk][j] = from_f32<T>(t[8 * kk + j]);
        };
        relayout(dsb, dsa);
        if constexpr (DEC) relayout(pb, pa);
      } else {
        // through the wave's LDS tile [position][route]
#pragma unroll
        for (int a = 0; a < 4; ++a)
          store4(tb + c * TBP + 8 * a + 4 * g, dS[4 * a], dS[4 * a + 1], dS[4 * a + 2], dS[4 * a + 3]);
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int j = 0; j < 8; ++j) dsa[kk][j] = tb[(16 * kk + 8 * g + j) * TBP + c];
        if constexpr (DEC) {
          __builtin_amdgcn_wave_barrier();
#pragma unroll
          for (int a = 0; a < 4; ++a)
            store4(tb + c * TBP + 8 * a + 4 * g, P[4 * a], P[4 * a + 1], P[4 * a + 2], P[4 * a + 3]);
          __builtin_amdgcn_wave_barrier();
#pragma unroll
          for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int j = 0; j < 8; ++j) pa[kk][j] = tb[(16 * kk + 8 * g + j) * TBP + c];
        }
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        f32x16 o, o2;
#pragma unroll
        for (int e = 0; e < 16; ++e) o[e] = o2[e] = 0.f;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          mma(o, dsa[kk], kt[kk][db]);
          if (DEC) mma(o2, pa[kk], gt[kk][db]);
        }
        if constexpr (D == 16) {
          // only columns c < 16 are real: lanes c >= 16 take rows 16 .. 31
          // (accumulator entries 8 .. 15) of column c - 16 by a swap of
          // 16-lane rows, so every lane adds two runs of 4 routes instead
          // of half the lanes adding four
          float v[8], u[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const auto so = __builtin_amdgcn_permlane16_swap(__float_as_uint(o[e]), __float_as_uint(o[e + 8]), false, false);
            v[e] = __uint_as_float(so[0]);
            if (DEC) {
              const auto s2 = __builtin_amdgcn_permlane16_swap(__float_as_uint(o2[e]), __float_as_uint(o2[e + 8]), false, false);
              u[e] = __uint_as_float(s2[0]);
            }
          }
          const int off = (c & 15) * SP + 32 * sb + (c & 16) + 4 * g;
#pragma unroll
          for (int a = 0; a < 2; ++a) {
            f32x4* pa4 = reinterpret_cast<f32x4*>(slot_a + off + 8 * a);
            f32x4 x = *pa4;
#pragma unroll
            for (int q = 0; q < 4; ++q) x[q] += v[4 * a + q];
            *pa4 = x;
            if (DEC) {
              f32x4* pg4 = reinterpret_cast<f32x4*>(slot_g + off + 8 * a);
              f32x4 y = *pg4;
#pragma unroll
              for (int q = 0; q < 4; ++q) y[q] += u[4 * a + q];
              *pg4 = y;
            }
          }
        } else if (32 * db + c < D) {
          float* sa = slot_a + (32 * db + c) * SP + 32 * sb + 4 * g;
          float* sg = slot_g + (32 * db + c) * SP + 32 * sb + 4 * g;
#pragma unroll
          for (int a = 0; a < 4; ++a) {
            f32x4 v = *reinterpret_cast<f32x4*>(sa + 8 * a);
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] += o[4 * a + q];
            *reinterpret_cast<f32x4*>(sa + 8 * a) = v;
            if (DEC) {
              f32x4 u = *reinterpret_cast<f32x4*>(sg + 8 * a);
#pragma unroll
              for (int q = 0; q < 4; ++q) u[q] += o2[4 * a + q];
              *reinterpret_cast<f32x4*>(sg + 8 * a) = u;
            }
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
      load_init(min(sb + 1, NS - 1), si, di);
    };
    ShortBlock<T, D, DEC> b0, b1;
    f32x16 si, di;
    load_short(b0, ash, gsh, asht, gsht, SB0, lane);
    load_init(0, si, di);
    for (int sb = 0; sb < NS; sb += 2) {
      load_short(b1, ash, gsh, asht, gsht, SB0 + min(sb + 1, NS - 1), lane);
      route_block(b0, sb, si, di);
      if (sb + 1 < NS) {  // wave-uniform
        load_short(b0, ash, gsh, asht, gsht, SB0 + min(sb + 2, NS - 1), lane);
        route_block(b1, sb + 1, si, di);
      }
    }
    // the next tile's staged rows (issued at this tile's start, ahead of all
    // its route-operand loads) have landed; waited for here, before this
    // tile's stores, so the wait covers loads only
    if (stg) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    // long-side results for this wave's 32 positions: rows d, column = lane
    if (nok) {
      const int64_t row = ((int64_t)b * p.Nl + n) * (int64_t)(p.H * D) + h * D;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int d = 32 * db + 8 * a + 4 * g;
          if (d < D) {
            float v[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = p.s * dk[db][4 * a + q];
            long_store(dout_b, static_cast<T*>(p.dout_b_lo), row + d, p.acc_b, v);
            if (!DEC) {
              float u[4];
#pragma unroll
              for (int q = 0; q < 4; ++q) u[q] = dv[db][4 * a + q];
              long_store(dout_g, static_cast<T*>(p.dout_g_lo), row + d, p.acc_g, u);
            }
          }
        }
    }
  }
  __syncthreads();
  // fixed-order sum of the waves' slots: this chunk's short-side partials
  const int64_t po = ((int64_t)bh * p.R + r) * p.Mp * D + (int64_t)32 * SB0 * D;
  for (int e = threadIdx.x; e < 32 * NS * D; e += blockDim.x) {
    const int m = e / D, d = e % D;  // m: route within the window
    float sa = 0.f, sg = 0.f;
    for (int w = 0; w < W; ++w) {
      const float* sw = reinterpret_cast<const float*>(smem) + w * slot_floats;
      sa += sw[d * SP + m];
      if (DEC) sg += sw[D * SP + d * SP + m];
    }
    p.part_a[po + e] = sa * p.s;
    if (DEC) p.part_g[po + e] = sg;
  }
}

// ---------------------------------------------------------------------------
// reductions and operand preparation
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_bwd_reduce(BwdReduceParams p) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n = (int64_t)p.O * p.M * p.D;
  if (i >= n) return;
  const int o = (int)(i / ((int64_t)p.M * p.D)), md = (int)(i % ((int64_t)p.M * p.D));
  float s = p.base ? p.base[i] : 0.f;
  const int64_t st = (int64_t)p.Mp * p.D;
  for (int q = 0; q < p.P; ++q) {
    s = sum_run(s, p.part0 + (((int64_t)q * p.O + o) * p.R0) * st + md, st, p.R0);
    if (p.part1) s = sum_run(s, p.part1 + (((int64_t)q * p.O + o) * p.R1) * st + md, st, p.R1);
  }
  p.out[i] = s;
}

// Source value src[o][m][d] of a prep job (m < M).
template <typename T>
__device__ __forceinline__ float prep_value(const BwdPrepJob& J, int M, int D, int o, int m, int d) {
  const int64_t i = ((int64_t)o * M + m) * D + d;
  return J.src_is_f32 ? static_cast<const float*>(J.src)[i] : to_f32(static_cast<const T*>(J.src)[i]);
}

template <typename T>
__global__ __launch_bounds__(256) void k_bwd_prep(BwdPrepParams p) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int D = p.D, DB = (D + 31) / 32, NS = p.Mp / 32;
  for (int jb = 0; jb < p.njobs; ++jb) {
    const BwdPrepJob& J = p.job[jb];
    const int64_t nrows = (int64_t)J.O * p.Mp;
    const int64_t nfl = J.tfrag ? (int64_t)J.O * NS * 2 * DB * 64 : 0;
    if (i < nrows) {
      // one padded row: T copy, c and the log2 normaliser, 8 channels at a
      // time (D is a multiple of 16)
      const int o = (int)(i / p.Mp), m = (int)(i % p.Mp);
      const int64_t si = ((int64_t)o * p.M + m) * D;
      float cs = 0.f;
      for (int d0 = 0; d0 < D; d0 += 8) {
        float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        if (m < p.M) {
          if (J.src_is_f32) load8(static_cast<const float*>(J.src) + si + d0, v);
          else load8(static_cast<const T*>(J.src) + si + d0, v);
          if (J.dot) {
            float w[8];
            load8(J.dot + si + d0, w);
#pragma unroll
            for (int j = 0; j < 8; ++j) cs += v[j] * w[j];
          }
        }
        if (J.rows) {
          const float rs = J.rows_scale != 0.f ? J.rows_scale : 1.f;
          float u[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) u[j] = v[j] * rs;
          store8(static_cast<T*>(J.rows) + i * D + d0, u);
        }
      }
      if (J.c) J.c[i] = cs;
      if (J.l2) J.l2[i] = m < p.M ? J.lse[(int64_t)o * p.M + m] * kLog2e : 0.f;
      return;
    }
    i -= nrows;
    if (i < nfl) {
      // one lane of a transposed fragment: [O][Mp / 32][2][DB][64][8]
      const int lane = (int)(i % 64);
      int64_t q = i / 64;
      const int db = (int)(q % DB); q /= DB;
      const int kk = (int)(q % 2); q /= 2;
      const int sb = (int)(q % NS);
      const int o = (int)(q / NS);
      const int g = lane >> 5, c = lane & 31, d = 32 * db + c;
      T* dst = static_cast<T*>(J.tfrag) + i * 8;
      for (int j = 0; j < 8; ++j) {
        const int m = 32 * sb + 16 * kk + acc_row16(g, j);
        dst[j] = from_f32<T>((m < p.M && d < D) ? prep_value<T>(J, p.M, D, o, m, d) : 0.f);
      }
      return;
    }
    i -= nfl;
  }
}

template <typename T, int D, bool DEC>
hipError_t attn_bwd_go(const AttnBwdParams& p, hipStream_t s) {
  const int W = attn_bwd_waves(D, p.nsb, p.Mp, DEC, (int)sizeof(T));
  const size_t lds = attn_bwd_lds_bytes(D, p.nsb, p.Mp, DEC, W, (int)sizeof(T));
  const void* fn = reinterpret_cast<const void*>(&k_attn_bwd<T, D, DEC>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  k_attn_bwd<T, D, DEC><<<(int64_t)p.B * p.H * p.R, 64 * W, lds, s>>>(p);
  return hipGetLastError();
}

}  // namespace

int attn_bwd_waves(int D, int nsb, int Mp, bool dec, int elem_bytes) {
  for (int w = 4; w >= 1; w /= 2)
    if (attn_bwd_lds_bytes(D, nsb, Mp, dec, w, elem_bytes) <= 160 * 1024) return w;
  return 0;
}

size_t attn_bwd_lds_bytes(int D, int nsb, int Mp, bool dec, int waves, int elem_bytes) {
  return (size_t)waves * attn_bwd_wave_bytes(D, nsb, dec, elem_bytes) + (dec ? 0 : 2 * sizeof(float) * (size_t)Mp);
}

int gemm_tile(int n) { return n >= 128 ? 128 : 64; }

template <typename T>
hipError_t launch_gemm(const GemmParams& p, hipStream_t s) {
  const int tm = gemm_tile(p.M), tn = gemm_tile(p.N);
  const bool one_tile = (p.N + tn - 1) / tn == 1 && (p.M + tm - 1) / tm == 1;
  const int nz = p.nprob > 1 && one_tile ? p.nprob * ((p.splits + 7) / 8 * 8) : p.nprob * p.splits;
  dim3 grid((p.N + tn - 1) / tn, (p.M + tm - 1) / tm, nz);
  if (tm == 128 && tn == 128) k_gemm<T, 128, 128><<<grid, 256, 0, s>>>(p);
  else if (tm == 128) k_gemm<T, 128, 64><<<grid, 256, 0, s>>>(p);
  else if (tn == 128) k_gemm<T, 64, 128><<<grid, 256, 0, s>>>(p);
  else k_gemm<T, 64, 64><<<grid, 256, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_sum_splits(const float* part, float* const* out, int64_t n, int splits, int nprob, hipStream_t s) {
  SumOuts o{};
  for (int i = 0; i < nprob && i < 5; ++i) o.out[i] = out[i];
  k_sum_splits<<<(unsigned)((n * nprob + 255) / 256), 256, 0, s>>>(part, o, n, splits, nprob);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_attn_bwd(const AttnBwdParams& p, int D, bool dec, hipStream_t s) {
  if (dec) {
    if (D == 16) return attn_bwd_go<T, 16, true>(p, s);
    if (D == 32) return attn_bwd_go<T, 32, true>(p, s);
    return attn_bwd_go<T, 64, true>(p, s);
  }
  if (D == 16) return attn_bwd_go<T, 16, false>(p, s);
  if (D == 32) return attn_bwd_go<T, 32, false>(p, s);
  return attn_bwd_go<T, 64, false>(p, s);
}

hipError_t launch_bwd_reduce(const BwdReduceParams& p, hipStream_t s) {
  const int64_t n = (int64_t)p.O * p.M * p.D;
  k_bwd_reduce<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

int64_t bwd_prep_items(const BwdPrepParams& p, int jb) {
  const BwdPrepJob& J = p.job[jb];
  const int DB = (p.D + 31) / 32;
  return (int64_t)J.O * p.Mp + (J.tfrag ? (int64_t)J.O * (p.Mp / 32) * 2 * DB * 64 : 0);
}

template <typename T>
hipError_t launch_bwd_prep(const BwdPrepParams& p, hipStream_t s) {
  int64_t n = 0;
  for (int jb = 0; jb < p.njobs; ++jb) n += bwd_prep_items(p, jb);
  k_bwd_prep<T><<<(unsigned)((n + 255) / 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

template hipError_t launch_gemm<float>(const GemmParams&, hipStream_t);
template hipError_t launch_gemm<__bf16>(const GemmParams&, hipStream_t);
template hipError_t launch_attn_bwd<float>(const AttnBwdParams&, int, bool, hipStream_t);
template hipError_t launch_attn_bwd<__bf16>(const AttnBwdParams&, int, bool, hipStream_t);
template hipError_t launch_bwd_prep<float>(const BwdPrepParams&, hipStream_t);
template hipError_t launch_bwd_prep<__bf16>(const BwdPrepParams&, hipStream_t);

}  // namespace flarepp
