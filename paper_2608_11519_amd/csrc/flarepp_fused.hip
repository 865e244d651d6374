// Fused kernels of the FLARE++ mixer forward for gfx950.
//
// The mixer reads X three times (the two encode calls and the decode each
// need a global reduction over all tokens before the next can start) and
// writes O once; the projections K, V, K~, V~ and the decoded tokens Y never
// reach HBM.  Each kernel recomputes the projection it needs from a 32-token
// tile of X with MFMA, directly in the operand layout of the routing MFMAs:
//
//  * key projection, out^T = W^T X^T (rows = channels, cols = tokens): lane
//    (c, g) receives token c and the channels of its accumulator rows.  The
//    weight columns of every 32-channel block are permuted (key_perm) so that
//    register r < 8 holds channel 8g + r and register 8 + r holds 16 + 8g + r:
//    exactly the A operand (keys x d) of the encode scores and the B operand
//    (d x tokens) of the decode scores.
//  * value projection, out = X W (rows = tokens, cols = channels): lane (c, g)
//    receives channel c for the tokens of its accumulator rows, which is the
//    key order the score tile hands to the value product.  No data movement.
//  * decode output: the normalised head outputs stay in registers as the B
//    operand of the merge O^T = W_O^T Y^T; the merge fragments read W_O rows
//    in the accumulator's row order (merge_row) instead of moving data.
//
// k_encode_fused  calls 1 and 2 (Sec. 2.2, Eqs. (8) and (10)): per (batch,
//                 32-channel head group, query group, token chunk) one wave;
//                 writes split-key partials (m, l, acc) per route.
// k_combine_par   exact merge of the partials (App. A.3, Eqs. (24)-(28)) in a
//                 fixed order, parallel over chunk slices.
// k_decode_fused  call 3 (Eq. (11)) and the merge with W_O (Fig. 1): per
//                 (batch, 256 tokens) one workgroup of 8 waves; the route
//                 operands of each head group and the W_O blocks are staged
//                 through LDS, double buffered.
#include "flarepp_device.hpp"
#include "flarepp_internal.hpp"

namespace flarepp {

constexpr int kFrag = 512;  // elements of one 64-lane x 8 fragment

// Channel (within a 32-channel block) placed at accumulator row rho of the
// key projection so that lane (c, g), register r holds channel 8g + r (r < 8)
// or 16 + 8g + (r - 8) (r >= 8).
__device__ __forceinline__ int key_perm(int rho) {
  return 16 * (rho >> 4) + 8 * ((rho >> 2) & 1) + 4 * ((rho & 15) >> 3) + (rho & 3);
}
// Input channel (within a 16-channel k step) of element j of a merge
// fragment in half g: the accumulator row order of the decode output.
__device__ __forceinline__ int merge_row(int g, int j) { return 8 * (j >> 2) + 4 * g + (j & 3); }

// ---------------------------------------------------------------------------
// Weight fragments of the fused path and the seed operand, one launch.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void k_prep_fused(PrepFusedParams p) {
  const int C = p.C, KS = C / 16;
  const int64_t per_w = (int64_t)C * C / 8;  // fragment lanes per weight
  const int64_t nseed = (int64_t)p.H * p.Mp * p.D;
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx < 5 * per_w) {
    const int w = (int)(idx / per_w);
    const int64_t f = idx % per_w;
    const int lane = (int)(f & 63), ks = (int)((f >> 6) % KS), cb = (int)((f >> 6) / KS);
    const int g = lane >> 5, c = lane & 31, mode = p.mode[w];
    const int col = 32 * cb + (mode == kFragKeyPerm ? key_perm(c) : c);
    const T* W = (const T*)p.w[w];
    T* out = (T*)p.wf[w] + f * 8;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = 16 * ks + (mode == kFragMerge ? merge_row(g, j) : 8 * g + j);
      out[j] = W[(int64_t)row * C + col];
    }
    return;
  }
  idx -= 5 * per_w;
  if (idx < nseed) {
    const int d = (int)(idx % p.D);
    const int m = (int)((idx / p.D) % p.Mp);
    const int h = (int)(idx / ((int64_t)p.D * p.Mp));
    const float v = m < p.M ? to_f32(((const T*)p.seeds)[((int64_t)h * p.M + m) * p.D + d]) : 0.f;
    ((T*)p.seeds_op)[idx] = from_f32<T>(v * p.qscale);
  }
}

// ---- small helpers -----------------------------------------------------------
template <typename T>
__device__ __forceinline__ typename Frag<T>::type cvt8(const f32x16& a, int off, float scale = 1.f) {
  typename Frag<T>::type r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = from_f32<T>(a[off + e] * scale);
  return r;
}
// The fragment of lane l ^ 16 (moves the upper 16 columns of each half down).
__device__ __forceinline__ bf16x8 xor16(const bf16x8& v) {
  typedef __attribute__((ext_vector_type(4))) int i32x4;
  i32x4 w = __builtin_bit_cast(i32x4, v);
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = __shfl_xor(w[i], 16, 64);
  return __builtin_bit_cast(bf16x8, w);
}
__device__ __forceinline__ f32x8 xor16(const f32x8& v) {
  f32x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = __shfl_xor(v[i], 16, 64);
  return r;
}
template <typename T>
__device__ __forceinline__ typename Frag<T>::type pick(bool a, const typename Frag<T>::type& x,
                                                       const typename Frag<T>::type& y) {
  typename Frag<T>::type r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = a ? x[e] : y[e];
  return r;
}

// ---------------------------------------------------------------------------
// Encode with the projection fused (calls 1 and 2).
// ---------------------------------------------------------------------------
template <typename T, int D, int KSC, int NQW>
__global__ __launch_bounds__(256) void k_encode_fused(EncFusedParams p) {
  using F = typename Frag<T>::type;
  constexpr int HPG = (D == 16) ? 2 : 1;  // heads per 32-channel group
  constexpr int GB = (D == 64) ? 2 : 1;   // 32-channel blocks per group
  constexpr int KS = D / 16, RB = (D + 31) / 32;
  constexpr bool ONES_ROW = (D == 16);
  constexpr int WELEMS = GB * KSC * kFrag;  // fragments of one weight slice
  __shared__ __attribute__((aligned(16))) T wlds[2 * WELEMS];

  const int lane = lane_id(), g = lane >> 5, c = lane & 31, wave = threadIdx.x >> 6;
  const int HG = p.H / HPG;
  const int ncg = (p.nchunks + 3) >> 2;
  int bid = blockIdx.x;
  const int cg = bid % ncg;
  bid /= ncg;
  const int qg = bid % p.qgroups;
  bid /= p.qgroups;
  const int hg = bid % HG;
  const int b = bid / HG;

  {  // the head group's key and value weight slices -> LDS
    constexpr int n16 = WELEMS * (int)sizeof(T) / 16;
    const uint4* sk = reinterpret_cast<const uint4*>((const T*)p.wkf + (int64_t)hg * WELEMS);
    const uint4* sv = reinterpret_cast<const uint4*>((const T*)p.wvf + (int64_t)hg * WELEMS);
    uint4* dst = reinterpret_cast<uint4*>(wlds);
    for (int i = threadIdx.x; i < n16; i += 256) {
      dst[i] = sk[i];
      dst[n16 + i] = sv[i];
    }
  }
  __syncthreads();
  const int r = cg * 4 + wave;
  if (r >= p.nchunks) return;  // no barrier below
  const T* wk_l = wlds;
  const T* wv_l = wlds + WELEMS;

  // ---- query operands of the wave's slots (slot = head-in-group x block) ----
  const int nslots = HPG * p.QB;
  F qf[NQW][KS];
  float qn = 0.f;
#pragma unroll
  for (int i = 0; i < NQW; ++i) {
    const int s = qg * NQW + i;
    const bool ok = s < nslots;
    const int h = hg * HPG + (ok ? s / p.QB : 0), qb = ok ? s % p.QB : 0;
    const T* qp = (const T*)p.q_op + (int64_t)b * p.q_sb + ((int64_t)h * p.Mp + qb * 32 + c) * D;
    float sq = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      qf[i][j] = ok ? load_frag(qp + 16 * j + 8 * g) : zero_frag<T>();
      sq += sumsq(qf[i][j]);
    }
    qn = fmaxf(qn, sq);
  }
  const float qmax2 = halfmax_sum_nonneg(qn);

  f32x16 acc[NQW][RB];
  float m[NQW], ls[NQW];
#pragma unroll
  for (int i = 0; i < NQW; ++i) {
    m[i] = -INFINITY;
    ls[i] = 0.f;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][rb][e] = 0.f;
  }
  bool fastok = true;

  const int k0 = r * p.chunk, k1 = min(p.N, k0 + p.chunk);
  const T* xb = (const T*)p.x + (int64_t)b * p.N * p.C;
  F xf[KSC];
  {
    const bool ok = k0 + c < k1;
#pragma unroll
    for (int ks = 0; ks < KSC; ++ks)
      xf[ks] = ok ? load_frag(xb + (int64_t)(k0 + c) * p.C + 16 * ks + 8 * g) : zero_frag<T>();
  }

  for (int t0 = k0; t0 < k1; t0 += 32) {
    const int nvalid = min(32, k1 - t0);
    // prefetch the next tile of X
    F xn[KSC];
    {
      const bool ok = t0 + 32 + c < k1;
#pragma unroll
      for (int ks = 0; ks < KSC; ++ks)
        xn[ks] = ok ? load_frag(xb + (int64_t)(t0 + 32 + c) * p.C + 16 * ks + 8 * g) : zero_frag<T>();
    }
    // key projection -> score A operands
    f32x16 ka[GB];
#pragma unroll
    for (int cb = 0; cb < GB; ++cb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) ka[cb][e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KSC; ++ks)
        mma(ka[cb], load_frag(wk_l + ((cb * KSC + ks) * 64 + lane) * 8), xf[ks]);
    }
    F kf[HPG][KS];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh)
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        const int fi = hh * KS + j;
        kf[hh][j] = cvt8<T>(ka[fi >> 1], 8 * (fi & 1));
      }
    // value projection -> value A operands (rows = channels)
    f32x16 va[GB];
#pragma unroll
    for (int cb = 0; cb < GB; ++cb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) va[cb][e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KSC; ++ks)
        mma(va[cb], xf[ks], load_frag(wv_l + ((cb * KSC + ks) * 64 + lane) * 8));
    }
    F vf[HPG][2][RB];
    if (ONES_ROW) {
      const F v0 = cvt8<T>(va[0], 0), v1 = cvt8<T>(va[0], 8);
      const F w0 = xor16(v0), w1 = xor16(v1);
      const F fill = (c == 16) ? fill_frag<T>(1.f) : zero_frag<T>();
      vf[0][0][0] = pick<T>(c < 16, v0, fill);
      vf[0][1][0] = pick<T>(c < 16, v1, fill);
      vf[HPG - 1][0][0] = pick<T>(c < 16, w0, fill);
      vf[HPG - 1][1][0] = pick<T>(c < 16, w1, fill);
    } else {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        vf[0][0][rb] = cvt8<T>(va[rb], 0);
        vf[0][1][rb] = cvt8<T>(va[rb], 8);
      }
    }
    float kmax2 = 0.f;
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) kmax2 = fmaxf(kmax2, frag_rows_max_sq<T, KS>(kf[hh]));
    const bool fast = fastok && (qmax2 * kmax2 <= p.fast_lim);

#pragma unroll
    for (int i = 0; i < NQW; ++i) {
      const int s = qg * NQW + i;
      if (s >= nslots) continue;
      f32x16 sc;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = 0.f;
      if (HPG == 1 || s < p.QB) {
#pragma unroll
        for (int j = 0; j < KS; ++j) mma(sc, kf[0][j], qf[i][j]);
        softmax_pv_tile<T, RB, ONES_ROW>(acc[i], m[i], ls[i], sc, vf[0], nvalid, fast, lane);
      } else {
#pragma unroll
        for (int j = 0; j < KS; ++j) mma(sc, kf[HPG - 1][j], qf[i][j]);
        softmax_pv_tile<T, RB, ONES_ROW>(acc[i], m[i], ls[i], sc, vf[HPG - 1], nvalid, fast, lane);
      }
    }
    if (!fast) {
      bool ok = true;
#pragma unroll
      for (int i = 0; i < NQW; ++i) ok = ok && (m[i] == 0.f || m[i] == -INFINITY);
      fastok = wave_all(ok);
    }
#pragma unroll
    for (int ks = 0; ks < KSC; ++ks) xf[ks] = xn[ks];
  }

  // ---- partials ----
  constexpr int NQ4 = ONES_ROW ? 2 : 4;
#pragma unroll
  for (int i = 0; i < NQW; ++i) {
    const int s = qg * NQW + i;
    if (s >= nslots) continue;
    const int h = hg * HPG + s / p.QB, qb = s % p.QB;
    const float l = softmax_denominator<RB, ONES_ROW>(acc[i], ls[i], lane);
    const int64_t pidx = (((int64_t)b * p.H + h) * p.nchunks + r) * p.Mp + qb * 32 + c;
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
  }
}

// ---------------------------------------------------------------------------
// Exact merge of split-key partials, parallel over chunk slices.  A block of
// 256 threads owns 16 rows; thread (row, rs) folds chunks rs, rs+16, ... in
// order, then the 16 slices of a row are folded pairwise (xor 1, 2, 4, 8).
// The pairwise fold is symmetric, so every slice ends with the same bits.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void k_combine_par(CombineParams p) {
  const int t = threadIdx.x, rs = t & 15;
  const int rows_per_bh = p.Mp / 16;
  const int64_t bh = blockIdx.x / rows_per_bh;
  const int qrow = (blockIdx.x % rows_per_bh) * 16 + (t >> 4);
  float m = -INFINITY, l = 0.f, a[D];
#pragma unroll
  for (int d = 0; d < D; ++d) a[d] = 0.f;
  for (int r = rs; r < p.R; r += 16) {
    const int64_t pidx = (bh * p.R + r) * p.Mp + qrow;
    const float mr = p.part_ml[pidx * 2];
    if (mr == -INFINITY) continue;
    const float lr = p.part_ml[pidx * 2 + 1];
    float ar[D];
#pragma unroll
    for (int d = 0; d < D; d += 4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(p.part_acc + pidx * D + d);
      ar[d] = v[0]; ar[d + 1] = v[1]; ar[d + 2] = v[2]; ar[d + 3] = v[3];
    }
    const float mn = fmaxf(m, mr);
    const float wa = __builtin_amdgcn_exp2f(m - mn), wb = __builtin_amdgcn_exp2f(mr - mn);
    l = l * wa + lr * wb;
#pragma unroll
    for (int d = 0; d < D; ++d) a[d] = a[d] * wa + ar[d] * wb;
    m = mn;
  }
#pragma unroll
  for (int k = 1; k < 16; k <<= 1) {
    const float mo = __shfl_xor(m, k, 64), lo = __shfl_xor(l, k, 64);
    float ao[D];
#pragma unroll
    for (int d = 0; d < D; ++d) ao[d] = __shfl_xor(a[d], k, 64);
    const float mn = fmaxf(m, mo);
    if (mn != -INFINITY) {
      const float wa = __builtin_amdgcn_exp2f(m - mn), wb = __builtin_amdgcn_exp2f(mo - mn);
      l = l * wa + lo * wb;
#pragma unroll
      for (int d = 0; d < D; ++d) a[d] = a[d] * wa + ao[d] * wb;
      m = mn;
    }
  }
  const bool valid = qrow < p.M;
  const float inv = (valid && l > 0.f) ? 1.f / l : 0.f;
#pragma unroll
  for (int d0 = 0; d0 < D; d0 += 16) {
    const int d = d0 + rs;
    float v = 0.f;
#pragma unroll
    for (int k = 0; k < D; ++k)
      if (k == d) v = a[k];
    const float out = v * inv;
    if (valid && p.out32) p.out32[(bh * p.M + qrow) * D + d] = out;
    if (p.q_op) ((T*)p.q_op)[(bh * p.Mp + qrow) * D + d] = from_f32<T>(out * p.qscale);
    if (p.z_op) ((T*)p.z_op)[(bh * D + d) * p.Mp + qrow] = from_f32<T>(out);
  }
  if (valid && p.lse && rs == 0) p.lse[bh * p.M + qrow] = 0.6931471805599453f * (m + __log2f(l));
}

// ---------------------------------------------------------------------------
// Decode with the key projection and the merge fused (call 3 + W_O).
// ---------------------------------------------------------------------------
// Waves (of 32 tokens) per decode workgroup: 8, or 4 at C = 256 where the
// resident X and Y fragments need more than 256 registers.
constexpr int dec_waves(int C) { return C >= 256 ? 4 : 8; }

// Issue the global -> LDS copy of decode stage s (see k_decode_fused) into
// buffer s & 1; completion is awaited with vmcnt before the next barrier.
template <typename T, int D, int KSC>
__device__ __forceinline__ void decode_stage_issue(const DecFusedParams& p, char* smem, int SE, int b,
                                                   int s) {
  constexpr int HPG = (D == 16) ? 2 : 1, GB = (D == 64) ? 2 : 1;
  constexpr int C = KSC * 16, HG = C / 32 / GB, WELEMS = GB * KSC * kFrag;
  constexpr int NT = 64 * dec_waves(C), per16 = 16 / (int)sizeof(T);
  const int Mp = p.Mp, nq = HPG * Mp * D;
  const int n16 = (s < HG ? WELEMS + 2 * nq : KSC * kFrag) / per16;
  const int wave = threadIdx.x >> 6;
  const int64_t h0 = (int64_t)b * p.H + (int64_t)s * HPG;
  char* dst = smem + (size_t)(s & 1) * SE * sizeof(T);
  for (int k = 0; k * NT < n16; ++k) {
    const int i = k * NT + threadIdx.x;
    if (i >= n16) continue;
    const int e = i * per16;
    const T* src;
    if (s >= HG) src = (const T*)p.wof + (int64_t)(s - HG) * KSC * kFrag + e;
    else if (e < WELEMS) src = (const T*)p.wkf + (int64_t)s * WELEMS + e;
    else if (e - WELEMS < nq) src = (const T*)p.q_op + h0 * Mp * D + (e - WELEMS);
    else src = (const T*)p.z_op + h0 * D * Mp + (e - WELEMS - nq);
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)(dst + (size_t)(k * NT + wave * 64) * 16),
                                     16, 0, 0);
  }
}

template <typename T, int D, int KSC>
__global__ __launch_bounds__(64 * dec_waves(16 * KSC)) void k_decode_fused(DecFusedParams p) {
  using F = typename Frag<T>::type;
  constexpr int HPG = (D == 16) ? 2 : 1, GB = (D == 64) ? 2 : 1;
  constexpr int KS = D / 16, RB = (D + 31) / 32;
  constexpr bool ONES_ROW = (D == 16);
  constexpr int C = KSC * 16, CB = C / 32, HG = CB / GB;
  constexpr int WELEMS = GB * KSC * kFrag;  // key weight slice of one head group
  constexpr int NW = dec_waves(C), NT = 64 * NW, TOK = 32 * NW;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  T* bufs = reinterpret_cast<T*>(smem);
  const int SE = p.stage_elems;

  const int lane = lane_id(), g = lane >> 5, c = lane & 31, wave = threadIdx.x >> 6;
  const int nblk = (p.N + TOK - 1) / TOK;
  const int b = blockIdx.x / nblk;
  const int xrow = (blockIdx.x % nblk) * TOK + wave * 32 + c;
  const bool xok = xrow < p.N;
  const int Mp = p.Mp;
  const int RT = Mp / 32;

  // stage s < HG: [key weight slice][q_op of the group's heads][z_op of them];
  // stage HG + cb: the W_O fragments of output block cb.  Stage s lives in
  // buffer s & 1 and is copied global -> LDS directly (16 bytes per lane).
  auto stage_issue = [&](int s) { decode_stage_issue<T, D, KSC>(p, smem, SE, b, s); };
  auto stage_wait = [&]() {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };

  stage_issue(0);
  F xf[KSC];
#pragma unroll
  for (int ks = 0; ks < KSC; ++ks)
    xf[ks] = xok ? load_frag((const T*)p.x + ((int64_t)b * p.N + xrow) * C + 16 * ks + 8 * g)
                 : zero_frag<T>();
  stage_wait();

  F yf[KSC];  // decoded tokens, merge B operands (16 channels per k step)
#pragma unroll
  for (int hg = 0; hg < HG; ++hg) {
    stage_issue(hg + 1);
    const T* sb = bufs + (hg & 1) * SE;
    f32x16 ka[GB];
#pragma unroll
    for (int cb = 0; cb < GB; ++cb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) ka[cb][e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KSC; ++ks) mma(ka[cb], load_frag(sb + ((cb * KSC + ks) * 64 + lane) * 8), xf[ks]);
    }
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      const int h = hg * HPG + hh;
      F kf[KS];
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        const int fi = hh * KS + j;
        kf[j] = cvt8<T>(ka[fi >> 1], 8 * (fi & 1));
      }
      const float qmax2 = frag_rows_max_sq<T, KS>(kf);
      const T* ql = sb + WELEMS + hh * Mp * D;
      const T* zl = sb + WELEMS + HPG * Mp * D + hh * D * Mp;
      f32x16 acc[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[rb][e] = 0.f;
      float m = -INFINITY, ls = 0.f;
      bool fastok = true;
      for (int rt = 0; rt < RT; ++rt) {
        F qa[KS];
#pragma unroll
        for (int j = 0; j < KS; ++j) qa[j] = load_frag(ql + (rt * 32 + c) * D + 16 * j + 8 * g);
        F zv[2][RB];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const int d = rb * 32 + c;
            if (d < D) {
              const T* zp = zl + d * Mp + rt * 32 + 16 * hf + 4 * g;
              zv[hf][rb] = join<T>(load_half(zp), load_half(zp + 8));
            } else {
              zv[hf][rb] = (ONES_ROW && c == 16) ? fill_frag<T>(1.f) : zero_frag<T>();
            }
          }
        const float kmax2 = frag_rows_max_sq<T, KS>(qa);
        const bool fast = fastok && (qmax2 * kmax2 <= p.fast_lim);
        f32x16 sc;
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
        for (int j = 0; j < KS; ++j) mma(sc, qa[j], kf[j]);
        softmax_pv_tile<T, RB, ONES_ROW>(acc, m, ls, sc, zv, min(32, p.M - rt * 32), fast, lane);
        if (!fast) fastok = wave_all(m == 0.f || m == -INFINITY);
      }
      const float inv = 1.f / softmax_denominator<RB, ONES_ROW>(acc, ls, lane);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
          if (rb * 32 + 16 * hf < D) yf[h * KS + 2 * rb + hf] = cvt8<T>(acc[rb], 8 * hf, inv);
      if (p.y && xok) {
        T* yp = (T*)p.y + ((int64_t)b * p.N + xrow) * C + h * D;
        constexpr int NQ4 = ONES_ROW ? 2 : 4;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int q = 0; q < NQ4; ++q)
            store4(yp + rb * 32 + 8 * q + 4 * g, acc[rb][4 * q] * inv, acc[rb][4 * q + 1] * inv,
                   acc[rb][4 * q + 2] * inv, acc[rb][4 * q + 3] * inv);
      }
    }
    stage_wait();
  }

  // ---- merge: O^T = W_O^T Y^T, one 32-channel output block per stage ----
#pragma unroll
  for (int cbo = 0; cbo < CB; ++cbo) {
    const int s = HG + cbo;
    if (cbo + 1 < CB) stage_issue(s + 1);
    const T* sb = bufs + (s & 1) * SE;
    f32x16 o;
#pragma unroll
    for (int e = 0; e < 16; ++e) o[e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KSC; ++ks) mma(o, load_frag(sb + (ks * 64 + lane) * 8), yf[ks]);
    if (xok) {
      T* op = (T*)p.o + ((int64_t)b * p.N + xrow) * C + 32 * cbo;
#pragma unroll
      for (int q = 0; q < 4; ++q) store4(op + 8 * q + 4 * g, o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]);
    }
    if (cbo + 1 < CB) stage_wait();
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T>
hipError_t launch_prep_fused(const PrepFusedParams& p, hipStream_t s) {
  const int64_t n = 5 * (int64_t)p.C * p.C / 8 + (int64_t)p.H * p.Mp * p.D;
  k_prep_fused<T><<<(unsigned)((n + 255) / 256), 256, 0, s>>>(p);
  return hipGetLastError();
}

template <typename T, int D, int KSC, int NQW>
static hipError_t enc_one(const EncFusedParams& p, unsigned grid, hipStream_t s) {
  if constexpr (NQW > enc_nqw_cap(sizeof(T), D, KSC) || enc_fused_lds(KSC * 16, D, sizeof(T)) > 65536) {
    return hipErrorInvalidValue;
  } else {
    k_encode_fused<T, D, KSC, NQW><<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
  }
}

template <typename T, int D, int KSC>
static hipError_t enc_nqw(const EncFusedParams& p, int nqw, unsigned grid, hipStream_t s) {
  switch (nqw) {
    case 1: return enc_one<T, D, KSC, 1>(p, grid, s);
    case 2: return enc_one<T, D, KSC, 2>(p, grid, s);
    case 4: return enc_one<T, D, KSC, 4>(p, grid, s);
    case 8: return enc_one<T, D, KSC, 8>(p, grid, s);
  }
  return hipErrorInvalidValue;
}

template <typename T, int D>
static hipError_t enc_ksc(const EncFusedParams& p, int nqw, unsigned grid, hipStream_t s) {
  switch (p.C) {
    case 64: return enc_nqw<T, D, 4>(p, nqw, grid, s);
    case 128: return enc_nqw<T, D, 8>(p, nqw, grid, s);
    case 256: return enc_nqw<T, D, 16>(p, nqw, grid, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_encode_fused(const EncFusedParams& p, int D, int nqw, hipStream_t s) {
  const int hpg = D == 16 ? 2 : 1;
  const int64_t grid = (int64_t)p.B * (p.H / hpg) * p.qgroups * ((p.nchunks + 3) / 4);
  switch (D) {
    case 16: return enc_ksc<T, 16>(p, nqw, (unsigned)grid, s);
    case 32: return enc_ksc<T, 32>(p, nqw, (unsigned)grid, s);
    case 64: return enc_ksc<T, 64>(p, nqw, (unsigned)grid, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_combine_par(const CombineParams& p, hipStream_t s) {
  const unsigned grid = (unsigned)(p.BH * (p.Mp / 16));
  switch (p.D) {
    case 16: k_combine_par<T, 16><<<grid, 256, 0, s>>>(p); break;
    case 32: k_combine_par<T, 32><<<grid, 256, 0, s>>>(p); break;
    case 64: k_combine_par<T, 64><<<grid, 256, 0, s>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int decode_stage_elems(int C, int D, int Mp) {
  const int hpg = D == 16 ? 2 : 1, gb = D == 64 ? 2 : 1;
  const int head_stage = gb * (C / 16) * kFrag + 2 * hpg * Mp * D;
  const int wo_stage = (C / 16) * kFrag;
  return head_stage > wo_stage ? head_stage : wo_stage;
}

bool decode_fused_fits(int C, int D, int Mp, int elem_bytes) {
  const size_t se = (size_t)decode_stage_elems(C, D, Mp) * elem_bytes;
  return 2 * se <= 160 * 1024;
}

template <typename T, int D, int KSC>
static hipError_t dec_launch(const DecFusedParams& p, hipStream_t s) {
  if constexpr (!dec_fused_ok(sizeof(T), D, KSC)) {
    return hipErrorInvalidValue;
  } else {
  constexpr int NW = dec_waves(16 * KSC);
  const unsigned grid = (unsigned)((int64_t)p.B * ((p.N + 32 * NW - 1) / (32 * NW)));
  const size_t lds = 2 * (size_t)p.stage_elems * sizeof(T);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_decode_fused<T, D, KSC>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  k_decode_fused<T, D, KSC><<<grid, 64 * NW, lds, s>>>(p);
  return hipGetLastError();
  }
}

template <typename T, int D>
static hipError_t dec_ksc(const DecFusedParams& p, hipStream_t s) {
  switch (p.C) {
    case 64: return dec_launch<T, D, 4>(p, s);
    case 128: return dec_launch<T, D, 8>(p, s);
    case 256: return dec_launch<T, D, 16>(p, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_decode_fused(const DecFusedParams& p, int D, hipStream_t s) {
  switch (D) {
    case 16: return dec_ksc<T, 16>(p, s);
    case 32: return dec_ksc<T, 32>(p, s);
    case 64: return dec_ksc<T, 64>(p, s);
  }
  return hipErrorInvalidValue;
}

template hipError_t launch_prep_fused<float>(const PrepFusedParams&, hipStream_t);
template hipError_t launch_prep_fused<__bf16>(const PrepFusedParams&, hipStream_t);
template hipError_t launch_encode_fused<float>(const EncFusedParams&, int, int, hipStream_t);
template hipError_t launch_encode_fused<__bf16>(const EncFusedParams&, int, int, hipStream_t);
template hipError_t launch_combine_par<float>(const CombineParams&, hipStream_t);
template hipError_t launch_combine_par<__bf16>(const CombineParams&, hipStream_t);
template hipError_t launch_decode_fused<float>(const DecFusedParams&, int, hipStream_t);
template hipError_t launch_decode_fused<__bf16>(const DecFusedParams&, int, hipStream_t);

}  // namespace flarepp
