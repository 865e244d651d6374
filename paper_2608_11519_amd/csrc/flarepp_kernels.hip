// HIP kernels of the FLARE++ mixer forward for gfx950.
//
// The mixer (Fig. 1; Sec. 3.2, Eqs. (7)-(11)) is: project K,V,K~,V~ = X W;
// Q = SDPA(Q~, K~, V~) and Z = SDPA(Q, K, V) with the softmax over the N
// tokens; Y = SDPA(K, Q, Z) with the softmax over the M routes; O = merge(Y) W_O.
//
// All three routing calls run through one kernel, k_route.  A "unit" (one
// wave) holds NQ blocks of 32 queries in registers and streams 32-key tiles:
//   S^T   = K_tile . Q^T             (MFMA, rows = keys, cols = queries)
//   P     = 2^(S^T - m)              (softmax numerators, log2 units)
//   out^T += [V^T ; 1 ; 0] . P        (MFMA; for D = 16 the row of ones
//                                     yields the softmax denominators)
// For the two encode calls the queries are the M routes and the keys are a
// chunk of the N tokens; each unit writes a partial (m, l, acc) that
// k_combine_par merges exactly in a fixed chunk order (App. A.2-A.3, Eqs. (19)-(28),
// with (m, l) carrying the log-normaliser L_r = m + log l).  For the decode the
// queries are 32-token blocks and the keys are all M routes; each unit writes
// normalised head outputs straight into Y[B][N][C].  The N x M scores never
// leave registers.  k_combine_par (flarepp_fused.hip) merges the partials.
//
// Scores are pre-scaled by log2(e)/sqrt(D) on the query operand (the route
// side), so the exponentials are bare v_exp_f32.  While the Cauchy-Schwarz
// bound |q.k| <= max|q| max|k| keeps every score within 64 (log2 units) of zero,
// no running maximum is needed (softmax is shift invariant); otherwise the
// tile falls back to the usual online-maximum update.
#include "flarepp_device.hpp"
#include "flarepp_internal.hpp"

namespace flarepp {

// ---------------------------------------------------------------------------
// Weight fragments: W [C][C] row-major (out = X W) -> per (column block cb,
// k step ks) one 64-lane fragment; lane l holds W[16ks + 8g + j][32cb + c].
// The same fragment is the A operand of O^T = W^T X^T and the B operand of
// O = X W.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void k_weight_frags(WeightFragParams p) {
  const int C = p.C, KS = C / 16;
  const int64_t per_w = (int64_t)(C / 32) * KS * 64;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= per_w * p.nw) return;
  const int w = (int)(idx / per_w);
  const int64_t f = idx % per_w;
  const int lane = (int)(f & 63), ks = (int)((f >> 6) % KS), cb = (int)((f >> 6) / KS);
  const T* W = (const T*)p.w[w];
  T* out = (T*)p.out[w] + f * 8;
  const int col = 32 * cb + (lane & 31), k0 = 16 * ks + 8 * (lane >> 5);
#pragma unroll
  for (int j = 0; j < 8; ++j) out[j] = W[(int64_t)(k0 + j) * C + col];
}

// ---------------------------------------------------------------------------
// Route-side operands from an fp32 (or storage-type) [B?][H][M][D] tensor:
//   q_op [B][H][Mp][D]  = src * qscale  (query operand of the encode calls and
//                                        key operand of the decode call)
//   z_op [B][H][D][Mp]  = src           (value operand of the decode call)
// Rows M..Mp-1 are zero.
// ---------------------------------------------------------------------------
template <typename Ts, typename T>
__global__ void k_route_prep(RoutePrepParams p) {
  const int64_t total = (int64_t)p.B * p.H * p.Mp * p.D;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int d = (int)(idx % p.D);
  const int m = (int)((idx / p.D) % p.Mp);
  const int64_t bh = idx / ((int64_t)p.D * p.Mp);
  const int b = (int)(bh / p.H), h = (int)(bh % p.H);
  float v = 0.f;
  if (m < p.M) v = to_f32(((const Ts*)p.src)[b * p.src_bstride + ((int64_t)h * p.M + m) * p.D + d]);
  if (p.q_op) ((T*)p.q_op)[(bh * p.Mp + m) * p.D + d] = from_f32<T>(v * p.qscale);
  if (p.z_op) ((T*)p.z_op)[(bh * p.D + d) * p.Mp + m] = from_f32<T>(v);
}

// ---------------------------------------------------------------------------
// Token-side values [B][H][N][D] -> d-major [B][H][D][Np], zero padded.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void k_dmajor(DmajorParams p) {
  const int64_t total = (int64_t)p.BH * p.D * p.Np;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int n = (int)(idx % p.Np);
  const int64_t bhd = idx / p.Np;
  const int d = (int)(bhd % p.D);
  const int64_t bh = bhd / p.D;
  T v = from_f32<T>(0.f);
  if (n < p.N) v = ((const T*)p.src)[(bh * p.N + n) * p.D + d];
  ((T*)p.dst)[idx] = v;
}

// ---------------------------------------------------------------------------
// Projection GEMM: out = X W for up to five weights.  One wave computes one
// 32-token x 32-column block.  Output layouts:
//   kHeadsTokenMajor [B][H][N][D]   (heads are contiguous D-column blocks)
//   kHeadsDMajor     [B][H][D][Np]  (zero padded to Np tokens)
//   kPlain           [B][N][C]
// ---------------------------------------------------------------------------
// One wave: 32 tokens of one weight's product, up to four 32-column output
// blocks at once (independent accumulators), the token fragments loaded once.
constexpr int kProjBlocks = 4;

// Lane (c, g) of a 32x32 result block holds rows 8 (j / 4) + 4 g + j % 4 of
// column c (j = 0..15): runs of 4 rows.  Swapping runs between the two lane
// halves (v_permlane32_swap; lanes c and c + 32 exchange) leaves lane (c, g)
// with rows 16 pr + 8 g .. + 7 in r[pr], pr = 0, 1: runs of 8 rows, one
// 16-byte (bf16) store each instead of two 8-byte ones, so a store
// instruction covers half as many memory segments.  All 64 lanes take part.
__device__ __forceinline__ void runs8(const f32x16& acc, float (&r)[2][8]) {
#pragma unroll
  for (int pr = 0; pr < 2; ++pr)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      // lanes 0-31 keep their rows 4 g + e and take the other half's; lanes
      // 32-63 take the other half's rows 8 + e and keep their own 12 + e
      const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[8 * pr + e]),
                                                      __float_as_uint(acc[8 * pr + 4 + e]), false, false);
      r[pr][e] = __uint_as_float(s[0]);
      r[pr][4 + e] = __uint_as_float(s[1]);
    }
}
__device__ __forceinline__ void store8(__bf16* p, const float (&v)[8]) {
  bf16x8 w;
#pragma unroll
  for (int i = 0; i < 8; ++i) w[i] = (__bf16)v[i];
  *reinterpret_cast<bf16x8*>(p) = w;
}
__device__ __forceinline__ void store8(float* p, const float (&v)[8]) {
  f32x4 a, b;
#pragma unroll
  for (int i = 0; i < 4; ++i) { a[i] = v[i]; b[i] = v[4 + i]; }
  reinterpret_cast<f32x4*>(p)[0] = a;
  reinterpret_cast<f32x4*>(p)[1] = b;
}

template <typename T, int NQ = kProjBlocks, int LAYOUT = -1>
__device__ __forceinline__ void proj_store(const ProjParams& p, int b, int n0, int w, int cg,
                                           const f32x16 (&acc)[NQ]);

// One unit: tokens [n0, n0 + 32) of batch entry b times column group cg of
// weight w, whose fragments start at wf (global memory or an LDS copy).
template <typename T>
__device__ __forceinline__ void proj_unit(const ProjParams& p, int b, int n0, int w, int cg, const T* wf) {
  using F = typename Frag<T>::type;
  const int lane = lane_id(), g = lane >> 5, c = lane & 31;
  const int CB = p.C / 32, KS = p.C / 16;
  const int layout = p.layout[w];
  const T* X = (const T*)p.x + ((int64_t)b * p.N) * p.C;
  const int xrow = n0 + c;
  const bool xok = xrow < p.N;
  f32x16 acc[kProjBlocks];
#pragma unroll
  for (int q = 0; q < kProjBlocks; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[q][r] = 0.f;
  // the operands of k step ks + 1 are loaded before the products of step ks;
  // rows past N load row N - 1 and are zeroed (the d-major layout stores them
  // as the zero padding)
  const T* xr = X + (int64_t)min(xrow, p.N - 1) * p.C + 8 * g;
  const T* wr = wf + (int64_t)cg * kProjBlocks * KS * 512 + lane * 8;
  const int nq = min(kProjBlocks, CB - cg * kProjBlocks);  // wave-uniform
  F xn = load_frag(xr), wn[kProjBlocks];
#pragma unroll
  for (int q = 0; q < kProjBlocks; ++q)
    if (q < nq) wn[q] = load_frag(wr + (int64_t)q * KS * 512);
  for (int ks = 0; ks < KS; ++ks) {
    const F xf = xok ? xn : zero_frag<T>();
    F wv[kProjBlocks];
#pragma unroll
    for (int q = 0; q < kProjBlocks; ++q) wv[q] = wn[q];
    if (ks + 1 < KS) {
      xn = load_frag(xr + 16 * (ks + 1));
#pragma unroll
      for (int q = 0; q < kProjBlocks; ++q)
        if (q < nq) wn[q] = load_frag(wr + ((int64_t)q * KS + ks + 1) * 512);
    }
#pragma unroll
    for (int q = 0; q < kProjBlocks; ++q) {
      if (q >= nq) break;  // wave-uniform
      if (layout == kHeadsDMajor) mma(acc[q], xf, wv[q]);   // rows = tokens, cols = channels
      else mma(acc[q], wv[q], xf);                          // rows = channels, cols = tokens
    }
  }
  proj_store<T>(p, b, n0, w, cg, acc);
}

// Stores the (up to) NQ result blocks acc of one unit (tokens [n0, n0 + 32)
// of batch entry b, column group cg of weight w) in weight w's layout, adding
// the residual for the plain layout when there is one.  LAYOUT is weight w's
// layout when known at compile time, else -1.
template <typename T, int NQ, int LAYOUT>
__device__ __forceinline__ void proj_store(const ProjParams& p, int b, int n0, int w, int cg,
                                           const f32x16 (&acc)[NQ]) {
  int lane = lane_id();
  // computed again at each call: kept from being hoisted out of a caller's
  // loops, where the per-lane store offsets would occupy registers throughout
  asm volatile("" : "+v"(lane));
  const int g = lane >> 5, c = lane & 31;
  const int CB = p.C / 32;
  const int layout = LAYOUT >= 0 ? LAYOUT : p.layout[w];
  const int xrow = n0 + c;
  const bool xok = xrow < p.N;
  T* out = (T*)p.out[w];
  const int D = p.D;
  // the residual of every block is loaded before the first store uses it
  const bool has_res = layout == kPlain && p.res && xok;
  Res16<T> res[NQ];
  if (has_res) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int cb = cg * NQ + q;
      if (cb >= CB) break;  // wave-uniform
      load_res16(res[q], (const T*)p.res + ((int64_t)b * p.N + xrow) * p.C + 32 * cb, g);
    }
  }
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int cb = cg * NQ + q;
    if (cb >= CB) break;  // wave-uniform
    if (layout == kHeadsDMajor) {
      // rows = tokens: two runs of 8 tokens per lane, 16-byte (bf16) stores
      float r[2][8];
      runs8(acc[q], r);
      const int col = 32 * cb + c, h = col / D, d = col % D;
      T* o = out + (((int64_t)b * p.H + h) * D + d) * p.Np + n0 + 8 * g;
      store8(o, r[0]);
      store8(o + 16, r[1]);
    } else if (layout == kPlain) {
      if (xok) store16(out + ((int64_t)b * p.N + xrow) * p.C + 32 * cb, acc[q], res[q], has_res, g);
    } else if (D % 8 == 0) {
      // rows = channels: two runs of 8 channels of one head per lane
      float r[2][8];
      runs8(acc[q], r);
      if (xok) {
#pragma unroll
        for (int pr = 0; pr < 2; ++pr) {
          const int col = 32 * cb + 16 * pr + 8 * g, h = col / D, d = col % D;
          store8(out + (((int64_t)b * p.H + h) * p.N + xrow) * D + d, r[pr]);
        }
      }
    } else if (xok) {
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = 32 * cb + 8 * r4 + 4 * g;
        const int h = col / D, d = col % D;
        store4(out + (((int64_t)b * p.H + h) * p.N + xrow) * D + d, acc[q][4 * r4], acc[q][4 * r4 + 1],
               acc[q][4 * r4 + 2], acc[q][4 * r4 + 3]);
      }
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_project(ProjParams p) {
  const int CB = p.C / 32, NB = p.Np / 32, CG = (CB + kProjBlocks - 1) / kProjBlocks;
  const int64_t u = (int64_t)blockIdx.x * 4 + wave_id();
  const int64_t total = (int64_t)p.B * NB * CG * p.nw;
  if (u >= total) return;
  const int cg = (int)(u % CG);
  const int w = (int)((u / CG) % p.nw);
  const int64_t bn = u / ((int64_t)CG * p.nw);
  proj_unit<T>(p, (int)(bn / NB), (int)(bn % NB) * 32, w, cg, (const T*)p.wf[w]);
}

// One unit of the persistent form: the tile's X fragments xf times weight w
// (fragments in LDS at wl), all CB = C / 32 column blocks, then the stores.
// The d-major layout takes result rows = tokens, the others rows = channels.
template <int KS, int LAYOUT>
__device__ __forceinline__ void proj_lds_unit(const ProjParams& p, int b, int n0, int w, const __bf16* wl,
                                              const bf16x8 (&xf)[KS]) {
  constexpr int CB = KS / 2;
  const __bf16* wr = wl + lane_id() * 8;
  f32x16 acc[CB];
#pragma unroll
  for (int q = 0; q < CB; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[q][r] = 0.f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int q = 0; q < CB; ++q) {
      const bf16x8 wv = load_frag(wr + (q * KS + ks) * 512);
      if (LAYOUT == kHeadsDMajor) mma(acc[q], xf[ks], wv);
      else mma(acc[q], wv, xf[ks]);
    }
  // issue order: the LDS reads of k step ks + 1 go out before the products
  // of step ks, and no further ahead (all of them hoisted would hold KS CB
  // fragments in registers)
  __builtin_amdgcn_sched_group_barrier(0x100, CB, 0);
#pragma unroll
  for (int ks = 1; ks < KS; ++ks) {
    __builtin_amdgcn_sched_group_barrier(0x100, CB, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, CB, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, CB, 0);
  proj_store<__bf16, CB, LAYOUT>(p, b, n0, w, 0, acc);
}

// Weight layout patterns of the persistent form (fixed at compile time so a
// tile's units are straight-line code): K, V (, K~, V~) as the mixer projects
// them, token-major outputs only, or one plain output (with residual).
enum ProjPattern { kPatKV = 0, kPatTok = 1, kPatPlain = 2 };

// Persistent form for bf16 when every weight's fragments fit in LDS together
// (C = 16 KS <= 128): a workgroup of 8 waves per CU copies them in once, then
// each wave walks 32-token tiles (tile = blockIdx.x * 8 + wave, + 8
// gridDim.x, ...).  A tile's rows of X stay in registers for all its units
// (KS fragments) and the next tile's rows are loaded while the current one is
// computed, so a wave keeps a whole tile's X reads in flight instead of one
// fragment per k step.  kPatKV: weights alternate token-major, d-major
// (nw = 2 or 4); kPatTok: nw token-major; kPatPlain: nw = 1, plain.
template <int KS, int PAT>
__global__ __launch_bounds__(512) void k_project_lds(ProjParams p) {
  using T = __bf16;
  using F = Frag<T>::type;
  constexpr int C = 16 * KS, CB = C / 32;  // one column group: CB <= kProjBlocks
  static_assert(CB >= 1 && CB <= kProjBlocks, "C = 32 .. 32 kProjBlocks");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  for (int w = 0; w < p.nw; ++w)
    copy_to_lds(p.wf[w], smem + (size_t)w * C * C * sizeof(T), C * C * (int)sizeof(T) / 16, 512);
  const int lane = lane_id(), g = lane >> 5, c = lane & 31;
  const int NB = p.Np / 32;
  const int64_t tiles = (int64_t)p.B * NB, stride = (int64_t)gridDim.x * 8;
  int64_t t = (int64_t)blockIdx.x * 8 + wave_id();
  const __bf16* wl = reinterpret_cast<const __bf16*>(smem);
  // rows past N load row N - 1 and are zeroed before use (the d-major layout
  // stores them as the zero padding)
  auto load_tile = [&](F (&xf)[KS], int64_t tile) {
    const int bb = (int)(tile / NB), row = min((int)(tile % NB) * 32 + c, p.N - 1);
    const T* xr = (const T*)p.x + ((int64_t)bb * p.N + row) * C + 8 * g;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) xf[ks] = load_frag(xr + 16 * ks);
  };
  // one tile: this tile's rows (loaded one tile earlier) are waited for
  // first (the empty asm reads them, so the wait sits here, ahead of the next
  // tile's loads, and not in the units), then the next tile's rows go out,
  // then every weight's unit
  auto tile = [&](F (&xf)[KS], F (&xn)[KS], int64_t tt) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("; x tile %0" : "+v"(xf[ks]));
    if (tt + stride < tiles) load_tile(xn, tt + stride);
    const int b = (int)(tt / NB), n0 = (int)(tt % NB) * 32;
    if (n0 + c >= p.N) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) xf[ks] = zero_frag<T>();
    }
    if constexpr (PAT == kPatKV) {
      proj_lds_unit<KS, kHeadsTokenMajor>(p, b, n0, 0, wl, xf);
      proj_lds_unit<KS, kHeadsDMajor>(p, b, n0, 1, wl + C * C, xf);
      if (p.nw == 4) {
        proj_lds_unit<KS, kHeadsTokenMajor>(p, b, n0, 2, wl + 2 * C * C, xf);
        proj_lds_unit<KS, kHeadsDMajor>(p, b, n0, 3, wl + 3 * C * C, xf);
      }
    } else if constexpr (PAT == kPatTok) {
      for (int w = 0; w < p.nw; ++w) proj_lds_unit<KS, kHeadsTokenMajor>(p, b, n0, w, wl + w * C * C, xf);
    } else {
      proj_lds_unit<KS, kPlain>(p, b, n0, 0, wl, xf);
    }
  };
  // two register sets, alternating (no copies between tiles)
  F xa[KS], xb[KS];
  if (t < tiles) load_tile(xa, t);
  lds_wait_barrier();
  // the first tile's rows are complete here; reading them in the empty asm
  // tells the compiler so, which keeps the loop's waits at the distance of a
  // whole tile of stores
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) asm volatile("; x tile %0" : "+v"(xa[ks]));
  while (t < tiles) {
    tile(xa, xb, t);
    t += stride;
    if (t >= tiles) break;
    tile(xb, xa, t);
    t += stride;
  }
}

// ---------------------------------------------------------------------------
// Routing attention (see the file comment).  Template parameters: storage
// type T, head width D, query blocks per unit NQ, and whether the call is the
// decode (softmax over routes, normalised output) or an encode (softmax over
// a chunk of tokens, partial output).
// ---------------------------------------------------------------------------
template <typename T, int D, int NQ, bool DECODE>
__global__ __launch_bounds__(256) void k_route(RouteParams p) {
  using F = typename Frag<T>::type;
  constexpr int KS = D / 16;            // 16-wide k steps of the score product
  constexpr int RB = (D + 31) / 32;     // 32-row blocks of the value product
  constexpr bool ONES_ROW = (D == 16);  // value row 16 is all ones -> row sums
  const int lane = lane_id(), g = lane >> 5, c = lane & 31;
  const int64_t u = (int64_t)blockIdx.x * 4 + wave_id();
  const int64_t total = (int64_t)p.B * p.H * p.nchunks * p.qgroups;
  if (u >= total) return;
  const int qg = (int)(u % p.qgroups);
  const int r = (int)((u / p.qgroups) % p.nchunks);
  const int64_t bh = u / ((int64_t)p.qgroups * p.nchunks);
  const int b = (int)(bh / p.H), h = (int)(bh % p.H);
  const int k0 = r * p.key_chunk;
  const int k1 = min(p.key_len, k0 + p.key_chunk);
  const int qb0 = qg * NQ;

  const T* ka = (const T*)p.ka + b * p.ka_sb + h * p.ka_sh;
  const T* va = (const T*)p.va + b * p.va_sb + h * p.va_sh;
  const T* qs = (const T*)p.qs + b * p.qs_sb + h * p.qs_sh;

  // ---- query operands, resident for the whole unit ----
  F qf[NQ][KS];
  float qn = 0.f;
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int row = (qb0 + i) * 32 + c;
    const bool ok = (qb0 + i) < p.nqb && row < p.qs_rows;
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      qf[i][j] = ok ? load_frag(qs + (int64_t)row * D + 16 * j + 8 * g) : zero_frag<T>();
      s += sumsq(qf[i][j]);
    }
    qn = fmaxf(qn, s);
  }
  const float qmax2 = halfmax_sum_nonneg(qn);

  // ---- softmax state ----
  f32x16 acc[NQ][RB];
  float m[NQ], ls[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    m[i] = -INFINITY;
    ls[i] = 0.f;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][rb][e] = 0.f;
  }
  bool fastok = true;  // every m is -inf or 0: the shift-free path is exact
  const float fast_lim = p.fast_lim;

  for (int t0 = k0; t0 < k1; t0 += 32) {
    const int nvalid = min(32, k1 - t0);
    // key operands: A[key][d] for the scores, A[d][key] for the values
    F kf[KS];
    const int krow = t0 + c;
    float kn = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      kf[j] = krow < p.ka_rows ? load_frag(ka + (int64_t)krow * D + 16 * j + 8 * g) : zero_frag<T>();
      kn += sumsq(kf[j]);
    }
    F vf[2][RB];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int d = rb * 32 + c;
        if (d < D) {
          const T* vp = va + (int64_t)d * p.va_ld + t0 + 16 * hf + 4 * g;
          vf[hf][rb] = join<T>(load_half(vp), load_half(vp + 8));
        } else {
          vf[hf][rb] = (ONES_ROW && c == 16) ? fill_frag<T>(1.f) : zero_frag<T>();
        }
      }
    const float kmax2 = halfmax_sum_nonneg(kn);
    const bool fast = fastok && uniform(qmax2 * kmax2 <= fast_lim);

#pragma unroll
    for (int i = 0; i < NQ; ++i) {
      if (qb0 + i >= p.nqb) continue;
      f32x16 s;
#pragma unroll
      for (int e = 0; e < 16; ++e) s[e] = 0.f;
#pragma unroll
      for (int j = 0; j < KS; ++j) mma(s, kf[j], qf[i][j]);
      softmax_pv_tile<T, RB, ONES_ROW>(acc[i], m[i], ls[i], s, vf, nvalid, fast, lane);
    }
    if (!fast) {
      bool ok = true;
#pragma unroll
      for (int i = 0; i < NQ; ++i) ok = ok && (m[i] == 0.f || m[i] == -INFINITY);
      fastok = wave_all(ok);
    }
  }

  // ---- epilogue ----
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    if (qb0 + i >= p.nqb) continue;
    const float l = softmax_denominator<RB, ONES_ROW>(acc[i], ls[i], lane);
    const int qrow = (qb0 + i) * 32 + c;
    constexpr int NQ4 = ONES_ROW ? 2 : 4;  // groups of 4 output rows per row block
    if (!DECODE) {
      const int64_t pidx = (bh * p.nchunks + r) * p.Mp + qrow;
      float* pa = p.part_acc + pidx * D;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int q = 0; q < NQ4; ++q)
          store4(pa + rb * 32 + 8 * q + 4 * g, acc[i][rb][4 * q], acc[i][rb][4 * q + 1],
                 acc[i][rb][4 * q + 2], acc[i][rb][4 * q + 3]);
      if (g == 0) {
        p.part_ml[pidx * 2] = m[i];
        p.part_ml[pidx * 2 + 1] = l;
      }
    } else if (qrow < p.qs_rows) {
      if (p.lse2 && g == 0) p.lse2[bh * p.qs_rows + qrow] = m[i] + __log2f(l);
      const float inv = 1.f / l;
      T* yp = (T*)p.y + (int64_t)b * p.y_sb + (int64_t)qrow * p.y_row + h * D;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int q = 0; q < NQ4; ++q)
          store4(yp + rb * 32 + 8 * q + 4 * g, acc[i][rb][4 * q] * inv, acc[i][rb][4 * q + 1] * inv,
                 acc[i][rb][4 * q + 2] * inv, acc[i][rb][4 * q + 3] * inv);
    }
  }
}

// ---------------------------------------------------------------------------
// Layer normalisation (the block's pre-norm), one wave per token: the row in
// registers (C / 64 values per lane), exact mean, then the variance of the
// centred values, both reduced over the wave.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int k = 32; k >= 1; k >>= 1) x += __shfl_xor(x, k, 64);
  return x;
}

// Layer norm of one token per LPT lanes: each lane holds NCH runs of 8
// channels (one 16- or 32-byte load each), so the row is read once, the two
// sums are shuffles over the token's lanes, and a wave normalises 64 / LPT
// tokens at a time.  Channel of lane li, run u: 8 (u LPT + li) + j.
template <typename T, int LPT, int NCH>
__global__ __launch_bounds__(256) void k_layernorm_vec(LayerNormParams p) {
  using F = typename Frag<T>::type;
  constexpr int TPW = 64 / LPT;
  const int lane = lane_id(), li = lane % LPT;
  F gm[NCH], bt[NCH];
#pragma unroll
  for (int u = 0; u < NCH; ++u) {
    gm[u] = load_frag((const T*)p.gamma + 8 * (u * LPT + li));
    bt[u] = load_frag((const T*)p.beta + 8 * (u * LPT + li));
  }
  const float inv_c = 1.f / (float)p.C;
  for (int64_t t0 = ((int64_t)blockIdx.x * 4 + wave_id()) * TPW; t0 < p.T; t0 += (int64_t)gridDim.x * 4 * TPW) {
    const int64_t row = min(t0 + lane / LPT, p.T - 1);  // past the end: a duplicate, not stored
    const T* x = (const T*)p.x + row * p.C;
    float v[NCH][8];
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const F f = load_frag(x + 8 * (u * LPT + li));
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        v[u][j] = to_f32(f[j]);
        s += v[u][j];
      }
    }
#pragma unroll
    for (int k = 1; k < LPT; k <<= 1) s += __shfl_xor(s, k, 64);
    const float mean = s * inv_c;
    float q = 0.f;
#pragma unroll
    for (int u = 0; u < NCH; ++u)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        v[u][j] -= mean;
        q += v[u][j] * v[u][j];
      }
#pragma unroll
    for (int k = 1; k < LPT; k <<= 1) q += __shfl_xor(q, k, 64);
    const float rstd = 1.f / sqrtf(q * inv_c + p.eps);
    if (p.mean && li == 0 && t0 + lane / LPT < p.T) {
      p.mean[row] = mean;
      p.rstd[row] = rstd;
    }
    if (t0 + lane / LPT < p.T) {
      T* y = (T*)p.y + row * p.C;
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        F o;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = from_f32<T>(v[u][j] * rstd * to_f32(gm[u][j]) + to_f32(bt[u][j]));
        *reinterpret_cast<F*>(y + 8 * (u * LPT + li)) = o;
      }
    }
  }
}

// Any C (a multiple of 32): one wave per token, the row read three times
// (the sum, the centred squares and the output; the later reads hit the
// cache).
template <typename T>
__global__ __launch_bounds__(256) void k_layernorm(LayerNormParams p) {
  const int lane = lane_id();
  const T* gm = (const T*)p.gamma;
  const T* bt = (const T*)p.beta;
  for (int64_t row = (int64_t)blockIdx.x * 4 + wave_id(); row < p.T; row += (int64_t)gridDim.x * 4) {
    const T* x = (const T*)p.x + row * p.C;
    float s = 0.f;
    for (int ch = lane; ch < p.C; ch += 64) s += to_f32(x[ch]);
    const float mean = wave_sum(s) / (float)p.C;
    float q = 0.f;
    for (int ch = lane; ch < p.C; ch += 64) {
      const float d = to_f32(x[ch]) - mean;
      q += d * d;
    }
    const float rstd = 1.f / sqrtf(wave_sum(q) / (float)p.C + p.eps);
    if (p.mean && lane == 0) {
      p.mean[row] = mean;
      p.rstd[row] = rstd;
    }
    T* y = (T*)p.y + row * p.C;
    for (int ch = lane; ch < p.C; ch += 64)
      y[ch] = from_f32<T>((to_f32(x[ch]) - mean) * rstd * to_f32(gm[ch]) + to_f32(bt[ch]));
  }
}

// Input gradient of the block's layer norm plus the residual, one wave per
// token: with g = dxn * gamma and xhat = (x - mean) rstd,
// dx = dO + rstd (g - mean_c(g) - xhat mean_c(g xhat)).
template <typename T>
__global__ __launch_bounds__(256) void k_layernorm_bwd_dx(LayerNormBwdParams p) {
  const int lane = lane_id();
  const T* gm = (const T*)p.gamma;
  for (int64_t row = (int64_t)blockIdx.x * 4 + wave_id(); row < p.T; row += (int64_t)gridDim.x * 4) {
    const T* x = (const T*)p.x + row * p.C;
    const float* dxn = p.dxn + row * p.C;
    const float mu = p.mean[row], rs = p.rstd[row];
    float sg = 0.f, sgx = 0.f;
    for (int ch = lane; ch < p.C; ch += 64) {
      const float g = dxn[ch] * to_f32(gm[ch]);
      sg += g;
      sgx += g * (to_f32(x[ch]) - mu) * rs;
    }
    const float mg = wave_sum(sg) / (float)p.C, mgx = wave_sum(sgx) / (float)p.C;
    const T* dO = (const T*)p.dO + row * p.C;
    float* dx = p.dx + row * p.C;
    for (int ch = lane; ch < p.C; ch += 64) {
      const float g = dxn[ch] * to_f32(gm[ch]);
      const float xh = (to_f32(x[ch]) - mu) * rs;
      dx[ch] = to_f32(dO[ch]) + rs * (g - mg - xh * mgx);
    }
  }
}

// Partial sums of dgamma and dbeta over a chunk of tokens: one thread per
// channel (coalesced across the block), tokens in order.
template <typename T>
__global__ __launch_bounds__(256) void k_layernorm_bwd_params(LayerNormBwdParams p) {
  const int ch = blockIdx.x * 256 + threadIdx.x;
  const int z = blockIdx.y;
  if (ch >= p.C) return;
  const int64_t t0 = (int64_t)z * p.chunk, t1 = min(p.T, t0 + p.chunk);
  float sg = 0.f, sb = 0.f;
  for (int64_t t = t0; t < t1; ++t) {
    const float d = p.dxn[t * p.C + ch];
    sg += d * (to_f32(((const T*)p.x)[t * p.C + ch]) - p.mean[t]) * p.rstd[t];
    sb += d;
  }
  p.part[(int64_t)z * p.C + ch] = sg;
  p.part[((int64_t)p.nchunks + z) * p.C + ch] = sb;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
static inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

template <typename T>
hipError_t launch_weight_frags(const WeightFragParams& p, hipStream_t s) {
  const int64_t n = (int64_t)(p.C / 32) * (p.C / 16) * 64 * p.nw;
  k_weight_frags<T><<<blocks_for(n, 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

template <typename Ts, typename T>
hipError_t launch_route_prep(const RoutePrepParams& p, hipStream_t s) {
  const int64_t n = (int64_t)p.B * p.H * p.Mp * p.D;
  k_route_prep<Ts, T><<<blocks_for(n, 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_dmajor(const DmajorParams& p, hipStream_t s) {
  const int64_t n = (int64_t)p.BH * p.D * p.Np;
  k_dmajor<T><<<blocks_for(n, 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_layernorm(const LayerNormParams& p, hipStream_t s) {
  // lanes per token for one run of 8 channels each (C = 32 .. 512), or 64
  // lanes with 2 .. 8 runs (C = 1024 .. 4096); other widths take k_layernorm
  const int runs = p.C / 8;
  auto grid = [&](int tpw) { return (unsigned)std::min<int64_t>((p.T + 4 * tpw - 1) / (4 * tpw), 1 << 16); };
  switch (p.C % 8 == 0 ? runs : 0) {
    case 4: k_layernorm_vec<T, 4, 1><<<grid(16), 256, 0, s>>>(p); break;
    case 8: k_layernorm_vec<T, 8, 1><<<grid(8), 256, 0, s>>>(p); break;
    case 16: k_layernorm_vec<T, 16, 1><<<grid(4), 256, 0, s>>>(p); break;
    case 32: k_layernorm_vec<T, 32, 1><<<grid(2), 256, 0, s>>>(p); break;
    case 64: k_layernorm_vec<T, 64, 1><<<grid(1), 256, 0, s>>>(p); break;
    case 128: k_layernorm_vec<T, 64, 2><<<grid(1), 256, 0, s>>>(p); break;
    case 256: k_layernorm_vec<T, 64, 4><<<grid(1), 256, 0, s>>>(p); break;
    case 512: k_layernorm_vec<T, 64, 8><<<grid(1), 256, 0, s>>>(p); break;
    default: k_layernorm<T><<<grid(1), 256, 0, s>>>(p); break;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_layernorm_bwd(const LayerNormBwdParams& p, hipStream_t s) {
  k_layernorm_bwd_dx<T><<<(unsigned)std::min<int64_t>((p.T + 3) / 4, 1 << 16), 256, 0, s>>>(p);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  k_layernorm_bwd_params<T><<<dim3((unsigned)((p.C + 255) / 256), (unsigned)p.nchunks), 256, 0, s>>>(p);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_project(const ProjParams& p, hipStream_t s) {
  // the persistent form: bf16, C = 64 or 128, every weight in LDS, and one
  // of its layout patterns
  int pat = -1;
  {
    bool kv = (p.nw == 2 || p.nw == 4), tok = true;
    for (int w = 0; w < p.nw; ++w) {
      kv = kv && p.layout[w] == ((w & 1) ? kHeadsDMajor : kHeadsTokenMajor);
      tok = tok && p.layout[w] == kHeadsTokenMajor;
    }
    pat = kv ? kPatKV : tok ? kPatTok : (p.nw == 1 && p.layout[0] == kPlain) ? kPatPlain : -1;
  }
  const size_t lds = (size_t)p.nw * p.C * p.C * sizeof(T);
  if (std::is_same<T, __bf16>::value && (p.C == 64 || p.C == 128) && lds <= 160 * 1024 && pat >= 0) {
    using Kern = void (*)(ProjParams);
    static const Kern kerns[2][3] = {
        {&k_project_lds<4, kPatKV>, &k_project_lds<4, kPatTok>, &k_project_lds<4, kPatPlain>},
        {&k_project_lds<8, kPatKV>, &k_project_lds<8, kPatTok>, &k_project_lds<8, kPatPlain>}};
    const Kern fn = kerns[p.C == 128][pat];
    int dev = 0, ncu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
      e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    const int64_t tiles = (int64_t)p.B * (p.Np / 32);
    const unsigned grid = (unsigned)std::min<int64_t>(blocks_for(tiles, 8), std::max(ncu, 1));
    hipLaunchKernelGGL(fn, dim3(grid), dim3(512), lds, s, p);
    return hipGetLastError();
  }
  const int64_t units = (int64_t)p.B * (p.Np / 32) * ((p.C / 32 + kProjBlocks - 1) / kProjBlocks) * p.nw;
  k_project<T><<<blocks_for(units, 4), 256, 0, s>>>(p);
  return hipGetLastError();
}

template <typename T, int D, bool DEC>
static hipError_t launch_route_d(const RouteParams& p, hipStream_t s) {
  const int64_t units = (int64_t)p.B * p.H * p.nchunks * p.qgroups;
  const unsigned nb = blocks_for(units, 4);
  constexpr int NQ = route_nq(D, DEC);
  k_route<T, D, NQ, DEC><<<nb, 256, 0, s>>>(p);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_route(const RouteParams& p, int D, bool decode, hipStream_t s) {
  switch (D) {
    case 16: return decode ? launch_route_d<T, 16, true>(p, s) : launch_route_d<T, 16, false>(p, s);
    case 32: return decode ? launch_route_d<T, 32, true>(p, s) : launch_route_d<T, 32, false>(p, s);
    case 64: return decode ? launch_route_d<T, 64, true>(p, s) : launch_route_d<T, 64, false>(p, s);
  }
  return hipErrorInvalidValue;
}

template hipError_t launch_weight_frags<float>(const WeightFragParams&, hipStream_t);
template hipError_t launch_weight_frags<__bf16>(const WeightFragParams&, hipStream_t);
template hipError_t launch_route_prep<float, float>(const RoutePrepParams&, hipStream_t);
template hipError_t launch_route_prep<float, __bf16>(const RoutePrepParams&, hipStream_t);
template hipError_t launch_route_prep<__bf16, __bf16>(const RoutePrepParams&, hipStream_t);
template hipError_t launch_dmajor<float>(const DmajorParams&, hipStream_t);
template hipError_t launch_dmajor<__bf16>(const DmajorParams&, hipStream_t);
template hipError_t launch_layernorm<float>(const LayerNormParams&, hipStream_t);
template hipError_t launch_layernorm<__bf16>(const LayerNormParams&, hipStream_t);
template hipError_t launch_layernorm_bwd<float>(const LayerNormBwdParams&, hipStream_t);
template hipError_t launch_layernorm_bwd<__bf16>(const LayerNormBwdParams&, hipStream_t);
template hipError_t launch_project<float>(const ProjParams&, hipStream_t);
template hipError_t launch_project<__bf16>(const ProjParams&, hipStream_t);
template hipError_t launch_route<float>(const RouteParams&, int, bool, hipStream_t);
template hipError_t launch_route<__bf16>(const RouteParams&, int, bool, hipStream_t);

}  // namespace flarepp
