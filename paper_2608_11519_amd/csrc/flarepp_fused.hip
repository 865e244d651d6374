// Fused kernels of the FLARE++ mixer forward for gfx950.
//
// The mixer reads X three times (the two encode calls and the decode each
// need a global reduction over all tokens before the next can start) and
// writes O once; the projections K, V, K~, V~ and the decoded tokens Y never
// reach HBM.  Each kernel recomputes the projection it needs from 32-token
// tiles of X with MFMA, directly in the operand layout of the routing MFMAs:
//
//  * key projection, out^T = W^T X^T (rows = channels, cols = tokens): lane
//    (c, g) receives token c and the channels of its accumulator rows.  The
//    weight columns of every 32-channel block are permuted (key_perm) so that
//    register r < 8 holds channel 8g + r and register 8 + r holds 16 + 8g + r:
//    exactly the A operand (keys x d) of the encode scores and the B operand
//    (d x tokens) of the decode scores.
//  * value projection, out = X W (rows = tokens, cols = channels): lane (c, g)
//    receives channel c for the tokens of its accumulator rows, which is the
//    key order the score tile hands to the value product.
//  * decode output: the normalised head outputs stay in registers as the B
//    operand of the merge O^T = W_O^T Y^T; the merge fragments read W_O rows
//    in the accumulator's row order (acc_row16) instead of moving data.
//
// Route operands (the seeds, Q(X) and Z) live in "fragment order" (see
// flarepp_internal.hpp): every lane reads 16 contiguous bytes, so operand
// loads from LDS or memory are free of bank conflicts.
//
// k_encode_fused  calls 1 and 2 (Sec. 3.2, Eqs. (8) and (10)); the fixed-
//                 query encode (Sec. 3.1, Eq. (5)).  A workgroup of W waves
//                 owns (batch, 32-channel head group, token chunk); each wave
//                 projects one 32-token sub-tile of the next super-tile into
//                 LDS while it runs its query blocks over the W sub-tiles of
//                 the current one.  Writes split-key partials (m, l, acc).
//                 The first call of a forward also converts the weights and
//                 seeds the later kernels read into fragment order.
// k_combine_par   exact merge of the partials (App. A.3, Eqs. (24)-(28)) in a
//                 fixed order, parallel over chunk slices; writes the next
//                 call's route operands.
// k_decode_fused  call 3 (Eq. (11)) and the merge with W_O (Fig. 1): per
//                 (batch, 32 * waves tokens) one workgroup; the route operands
//                 of each head group and the W_O blocks are staged through LDS
//                 (direct global -> LDS copies), double buffered.
#include <algorithm>
#include <type_traits>

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

// ---- small helpers -----------------------------------------------------------
template <typename T>
__device__ __forceinline__ typename Frag<T>::type cvt8(const f32x16& a, int off, float scale = 1.f) {
  typename Frag<T>::type r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = from_f32<T>(a[off + e] * scale);
  return r;
}
template <typename T>
__device__ __forceinline__ void store_frag(T* p, const typename Frag<T>::type& v) {
  *reinterpret_cast<typename Frag<T>::type*>(p) = v;
}

// ---------------------------------------------------------------------------
// One item of the fused path's preparation: a lane of a weight fragment, a
// lane of the seed operand (scaled, in q fragment order, seed_copies copies)
// or, with qnorm2, one route-norm bound of the seed operand for the decode
// (the fixed-query path, where the seeds are the decode's routes).  The first
// combine of a forward runs them, spread over its threads: prep_load issues
// an item's loads, prep_store writes it once the combine's own work is done.
// ---------------------------------------------------------------------------
int64_t prep_fused_items(const PrepFusedParams& p) {
  return p.nw * (int64_t)p.C * p.C / 8 + (int64_t)p.seed_copies * p.H * (p.Mp / 32) * (p.D / 16) * 64 +
         (p.qnorm2 ? (int64_t)p.seed_copies * p.H * (p.Mp / 4) : 0);
}

template <typename T>
__device__ __forceinline__ typename Frag<T>::type prep_load(const PrepFusedParams& p, int64_t idx) {
  const int C = p.C, KS = C / 16;
  const int64_t per_w = (int64_t)C * C / 8;  // fragment lanes per weight
  const int QB = p.Mp / 32, DS = p.D / 16;
  const int64_t nseed = (int64_t)p.H * QB * DS * 64;
  typename Frag<T>::type v = zero_frag<T>();
  if (idx < p.nw * per_w) {  // a weight fragment lane
    const int w = (int)(idx / per_w);
    const int64_t f = idx % per_w;
    const int lane = (int)(f & 63), ks = (int)((f >> 6) % KS), cb = (int)((f >> 6) / KS);
    const int g = lane >> 5, c = lane & 31, mode = p.mode[w];
    const int col = 32 * cb + (mode == kFragKeyPerm ? key_perm(c) : c);
    const T* W = (const T*)p.w[w];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = 16 * ks + (mode == kFragMerge || mode == kFragMergeHg ? acc_row16(g, j) : 8 * g + j);
      v[j] = W[(int64_t)row * C + col];
    }
    return v;
  }
  idx -= p.nw * per_w;
  if (idx < p.seed_copies * nseed) {  // a seed operand lane, scaled
    const int64_t si = idx % nseed;
    const int lane = (int)(si & 63), js = (int)((si >> 6) % DS);
    const int qb = (int)((si >> 6) / DS % QB), h = (int)((si >> 6) / DS / QB);
    const int g = lane >> 5, m = 32 * qb + (lane & 31);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float x = m < p.M ? to_f32(((const T*)p.seeds)[((int64_t)h * p.M + m) * p.D + 16 * js + 8 * g + j]) : 0.f;
      v[j] = from_f32<T>(x * p.qscale);
    }
  }
  return v;
}

template <typename T>
__device__ __forceinline__ void prep_store(const PrepFusedParams& p, int64_t idx, const typename Frag<T>::type& v) {
  const int C = p.C, KS = C / 16;
  const int64_t per_w = (int64_t)C * C / 8;
  const int QB = p.Mp / 32, DS = p.D / 16;
  const int64_t nseed = (int64_t)p.H * QB * DS * 64;
  if (idx < p.nw * per_w) {
    const int w = (int)(idx / per_w);
    const int64_t f = idx % per_w;
    int64_t fo = f;
    if (p.mode[w] == kFragMergeHg) {  // [head group][output block][k step in group][64][8]
      const int lane = (int)(f & 63), ks = (int)((f >> 6) % KS), cb = (int)((f >> 6) / KS);
      const int kpg = p.D == 64 ? 4 : 2, CB = C / 32;
      fo = ((int64_t)((ks / kpg) * CB + cb) * kpg + ks % kpg) * 64 + lane;
    }
    store_frag<T>((T*)p.wf[w] + fo * 8, v);
    return;
  }
  idx -= p.nw * per_w;
  if (idx < p.seed_copies * nseed) {
    store_frag<T>((T*)p.seeds_op + idx * 8, v);
    return;
  }
  idx -= p.seed_copies * nseed;
  if (p.qnorm2 && idx < (int64_t)p.seed_copies * p.H * (p.Mp / 4)) {
    // max over routes 4i .. 4i+3 of |scaled q|^2 of the rounded operand
    const int64_t per = (int64_t)p.H * (p.Mp / 4);
    const int h = (int)(idx % per / (p.Mp / 4)), i = (int)(idx % (p.Mp / 4));
    float n2 = 0.f;
    for (int m = 4 * i; m < min(4 * i + 4, p.M); ++m) {
      float s = 0.f;
      for (int d = 0; d < p.D; ++d) {
        const float q = to_f32(from_f32<T>(to_f32(((const T*)p.seeds)[((int64_t)h * p.M + m) * p.D + d]) * p.qscale));
        s = __builtin_fmaf(q, q, s);
      }
      n2 = fmaxf(n2, s);
    }
    p.qnorm2[idx] = n2;
  }
}

// ---------------------------------------------------------------------------
// Encode with the projection fused (calls 1 and 2).
// ---------------------------------------------------------------------------
template <int D> struct EncShape {
  static constexpr int HPG = (D == 16) ? 2 : 1;  // heads per 32-channel group
  static constexpr int GB = (D == 64) ? 2 : 1;   // 32-channel blocks per group
  static constexpr int KS = D / 16, RB = (D + 31) / 32;
  static constexpr int KFR = HPG * KS;           // key fragments per sub-tile
  static constexpr int VFR = HPG * 2 * RB;       // value-operand fragments per sub-tile
  static constexpr int TILE = (KFR + VFR) * kFrag;
};

size_t enc_fused_lds_bytes(int C, int D, int waves, int elem_bytes) {
  const int gb = D == 64 ? 2 : 1, hpg = D == 16 ? 2 : 1, rb = (D + 31) / 32;
  const size_t welems = (size_t)gb * (C / 16) * kFrag;
  const size_t tile = (size_t)(hpg * (D / 16) + hpg * 2 * rb) * kFrag;
  return (2 * welems + 2 * waves * tile) * elem_bytes + 2 * waves * hpg * sizeof(float);
}

// LDS layout of one projected 32-token sub-tile:
//   key fragments (hh, js)          [KFR][64 lanes][8]: lane (c, g) = token c,
//                                    dims 16 js + 8 g .. + 7 of head hh
//   value operands (hh, rb, hf)     [VFR][64 lanes][8]: the A operand of the
//                                    value product for keys 16 hf .. 16 hf + 15
//                                    (in the score tile's row order); lane
//                                    (c, g) = channel 32 rb + c of head hh.
//                                    For D = 16 rows 16 .. 31 are constant
//                                    (row 16 ones: the denominators, the rest
//                                    zeros) and are written once.
template <typename T, int D, int KSC, int NQW, int W>
__global__ __launch_bounds__(64 * W) void k_encode_fused(EncFusedParams p) {
  using F = typename Frag<T>::type;
  using S = EncShape<D>;
  constexpr int HPG = S::HPG, GB = S::GB, KS = S::KS, RB = S::RB, KFR = S::KFR, TILE = S::TILE;
  constexpr bool ONES_ROW = (D == 16);
  constexpr int WELEMS = GB * KSC * kFrag;  // one weight slice of the head group
  constexpr int STEP = 32 * W;              // tokens per super-tile
  extern __shared__ __attribute__((aligned(16))) char smem[];
  T* wk_l = reinterpret_cast<T*>(smem);
  T* wv_l = wk_l + WELEMS;
  T* tiles = wv_l + WELEMS;  // [2][W][TILE]
  float* kmx = reinterpret_cast<float*>(tiles + 2 * W * TILE);  // [2][W][HPG]

  const int lane = lane_id(), g = lane >> 5, c = lane & 31, wave = wave_id();
  const int HG = p.H / HPG, G = HG * p.qgroups;
  // blocks of one token chunk (all head and query groups) share an XCD
  const int bid = blockIdx.x;
  const int64_t chunk_id = (int64_t)(bid >> 3) / G * 8 + (bid & 7);
  if (chunk_id >= (int64_t)p.B * p.nchunks) return;  // whole block, before any barrier
  const int hgq = (bid >> 3) % G;
  const int hg = hgq / p.qgroups, qg = hgq % p.qgroups;
  const int b = (int)(chunk_id / p.nchunks), r = (int)(chunk_id % p.nchunks);

  // The head group's weight slices in LDS, in fragment order: copied from the
  // fragments, or gathered from the row-major weights (key projection with
  // its columns key-permuted); the gathered lanes are written to LDS after
  // the route and X loads are issued.
  constexpr int WL = GB * KSC * 64, WPT = (WL + 64 * W - 1) / (64 * W);  // lanes, per thread
  F wkg[WPT], wvg[WPT];
  if (p.wk_raw) {
    const T* Wk = (const T*)p.wk_raw;
    const T* Wv = (const T*)p.wv_raw;
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int i = u * 64 * W + threadIdx.x;
      if (i < WL) {
        const int cb = hg * GB + i / (KSC * 64), ks = (i / 64) % KSC, ln = i % 64, gg = ln >> 5, cc = ln & 31;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int64_t row = (int64_t)(16 * ks + 8 * gg + j) * p.C + 32 * cb;
          wkg[u][j] = Wk[row + key_perm(cc)];
          wvg[u][j] = Wv[row + cc];
        }
      }
    }
  } else {
    copy_to_lds((const T*)p.wkf + (int64_t)hg * WELEMS, smem, WELEMS * (int)sizeof(T) / 16, 64 * W);
    copy_to_lds((const T*)p.wvf + (int64_t)hg * WELEMS, smem + WELEMS * sizeof(T), WELEMS * (int)sizeof(T) / 16,
                64 * W);
  }
  if constexpr (ONES_ROW) {  // constant rows 16 .. 31 of every value operand
    constexpr int NCONST = 2 * W * S::VFR * 32;
    for (int i = threadIdx.x; i < NCONST; i += 64 * W) {
      const int rr = i & 15, gg = (i >> 4) & 1, f = i >> 5;  // f = (buf * W + j) * VFR + vf
      T* dst = tiles + (f / S::VFR) * TILE + (KFR + f % S::VFR) * kFrag + (16 + rr + 32 * gg) * 8;
      store_frag<T>(dst, rr == 0 ? fill_frag<T>(1.f) : zero_frag<T>());
    }
  }

  // ---- this wave's query slots (slot = head-in-group x 32-query block); the
  // host makes every wave's slots belong to one head ----
  const int nslots = HPG * p.QB;
  const int slot0 = (qg * W + wave) * NQW;
  const int hh = HPG == 1 ? 0 : __builtin_amdgcn_readfirstlane(min(slot0, nslots - 1) / p.QB);
  F qf[NQW][KS];
#pragma unroll
  for (int i = 0; i < NQW; ++i) {
    const int s = slot0 + i;
    const bool ok = s < nslots;
    const int qb = ok ? s % p.QB : 0;
    if (p.seeds_raw) {  // the learned seeds, shared by the batch, scaled here
      const int m = 32 * qb + c;
      const T* sp = (const T*)p.seeds_raw + ((int64_t)(hg * HPG + hh) * p.M + m) * D;
#pragma unroll
      for (int js = 0; js < KS; ++js) {
        F v = zero_frag<T>();
        if (ok && m < p.M) {
          const F raw = load_frag(sp + 16 * js + 8 * g);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = from_f32<T>(to_f32(raw[e]) * p.qscale);
        }
        qf[i][js] = v;
      }
    } else {
      const T* qp = (const T*)p.q_op + (int64_t)b * p.q_sb + (int64_t)(hg * HPG + hh) * p.Mp * D;
#pragma unroll
      for (int js = 0; js < KS; ++js)
        qf[i][js] = ok ? load_frag(qp + ((int64_t)(qb * KS + js) * 64 + lane) * 8) : zero_frag<T>();
    }
  }

  f32x16 acc[NQW][RB];
  float m[NQW], ls[NQW];
#pragma unroll
  for (int i = 0; i < NQW; ++i) {
    m[i] = 0.f;  // the shift of the shift-free phase
    ls[i] = 0.f;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][rb][e] = 0.f;
  }

  const int k0 = r * p.chunk, k1 = min(p.N, k0 + p.chunk);
  const T* xb = (const T*)p.x + (int64_t)b * p.N * p.C;
  // X rows past the chunk are clamped to its last row: their keys and values
  // duplicate a real token's (masked out of the softmax, and never above the
  // key norm bound), and every load is unconditional, so the compiler can
  // count the loads in flight.  Each super-tile's rows are requested one
  // super-tile ahead and stay in flight across the LDS barriers.
  F xf[KSC];
  auto load_x = [&](int t) __attribute__((always_inline)) {
    const int row = min(t + 32 * wave + c, k1 - 1);
#pragma unroll
    for (int ks = 0; ks < KSC; ++ks) xf[ks] = load_frag(xb + (int64_t)row * p.C + 16 * ks + 8 * g);
  };
  asm volatile("" ::: "memory");  // the weight copies and route loads are issued first
  load_x(k0);
  if (p.wk_raw) {
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int i = u * 64 * W + threadIdx.x;
      if (i < WL) {
        store_frag<T>(wk_l + i * 8, wkg[u]);
        store_frag<T>(wv_l + i * 8, wvg[u]);
      }
    }
  }
  // weight slices and constant rows in LDS (every load but the X rows)
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(KSC) : "memory");
  lds_barrier();
  __builtin_amdgcn_sched_barrier(0);  // the norms below must not wait for the X loads
  float qn = 0.f;
#pragma unroll
  for (int i = 0; i < NQW; ++i) {
    float sq = 0.f;
#pragma unroll
    for (int js = 0; js < KS; ++js) sq += sumsq(qf[i][js]);
    qn = fmaxf(qn, sq);
  }
  const float qmax2 = halfmax_sum_nonneg(qn);

  // Projection of this wave's 32-token sub-tile of a super-tile: K and V of
  // the head group accumulate over the KSC k-steps of X (xf).  Each k-step
  // is issued after one route tile of the previous super-tile, so the matrix
  // work and the X traffic run beside the softmax; xf[ks] is refilled with
  // the rows of the super-tile after that right after its last use, which
  // gives every X load a whole super-tile to arrive.
  f32x16 ka[GB], va[GB];
  auto proj_zero = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int cb = 0; cb < GB; ++cb)
#pragma unroll
      for (int e = 0; e < 16; ++e) { ka[cb][e] = 0.f; va[cb][e] = 0.f; }
  };
  auto proj_step = [&](int ks, int trefill) __attribute__((always_inline)) {
#pragma unroll
    for (int cb = 0; cb < GB; ++cb) {
      const int fo = ((cb * KSC + ks) * 64 + lane) * 8;
      mma(ka[cb], load_frag(wk_l + fo), xf[ks]);
      mma(va[cb], xf[ks], load_frag(wv_l + fo));
    }
    const int row = min(trefill + 32 * wave + c, k1 - 1);
    xf[ks] = load_frag(xb + (int64_t)row * p.C + 16 * ks + 8 * g);
  };
  // the projected sub-tile into LDS buffer buf, with its key norm bound
  auto proj_store = [&](int buf) __attribute__((always_inline)) {
    T* tl = tiles + (buf * W + wave) * TILE;
#pragma unroll
    for (int h2 = 0; h2 < HPG; ++h2) {
      F kf[KS];
#pragma unroll
      for (int js = 0; js < KS; ++js) {
        const int fi = h2 * KS + js;
        kf[js] = cvt8<T>(ka[fi >> 1], 8 * (fi & 1));
        store_frag<T>(tl + fi * kFrag + lane * 8, kf[js]);
      }
      const float kb = frag_rows_max_sq<T, KS>(kf);
      if (lane == 0) kmx[(buf * W + wave) * HPG + h2] = kb;
    }
    if constexpr (ONES_ROW) {  // channel c -> row c % 16 of head c / 16's operand
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
        store_frag<T>(tl + (KFR + (c >> 4) * 2 + hf) * kFrag + ((c & 15) + 32 * g) * 8, cvt8<T>(va[0], 8 * hf));
    } else {
#pragma unroll
      for (int cb = 0; cb < GB; ++cb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
          store_frag<T>(tl + (KFR + 2 * cb + hf) * kFrag + lane * 8, cvt8<T>(va[cb], 8 * hf));
    }
  };

  // the first super-tile is projected before any route tile
  proj_zero();
#pragma unroll
  for (int ks = 0; ks < KSC; ++ks) proj_step(ks, k0 + STEP);
  proj_store(0);
  lds_barrier();

  // Run the wave's query slots over every sub-tile of the super-tile at t0
  // (LDS buffer it & 1): shift-free (SF) or with the online maximum; MASK
  // only for the last, partial super-tile of a chunk.  Every wave runs all
  // NQW slots: a slot past the last query block holds a zero query (its
  // tiles are wasted work, its partial is never stored), and the waves of a
  // workgroup meet at every super-tile anyway, so no tile sequence branches
  // per slot.  Unmasked runs also project the super-tile after this one (the
  // k-steps spread over the NT route tiles); after the last full super-tile
  // of a chunk without a tail that projection is of clamped rows and unused.
  constexpr int NT = W * NQW;
  auto consume = [&](auto sf, auto mask, int it, int t0) __attribute__((always_inline)) {
    constexpr bool SF = decltype(sf)::value, MASK = decltype(mask)::value;
    const int buf = it & 1;
    if (!MASK) proj_zero();
    auto hooks = [&](int n) __attribute__((always_inline)) {
      if constexpr (!MASK) {
#pragma unroll
        for (int ks = n * KSC / NT; ks < (n + 1) * KSC / NT; ++ks) proj_step(ks, t0 + 2 * STEP);
      }
    };
    if constexpr (!MASK && SF) {
      // Shift-free tiles n = j * NQW + i (sub-tile j, slot i), software
      // pipelined so that every MFMA is issued between groups of
      // exponentials whose inputs are long ready (a wave issues in order: an
      // MFMA waiting on the P it was just given, or on the busy matrix pipe,
      // stalls the exponentials behind it).  Per tile n, five phases:
      //   0: score MFMA of tile n + 1; LDS reads for tiles n + 1 and n + 2;
      //      2^s of scores 0..3
      //   1: value MFMAs of tile n - 1, keys 0..15; 2^s 4..7; pack P 0..7
      //   2: key-projection MFMAs (hook k-steps); 2^s 8..11
      //   3: value MFMAs of tile n - 1, keys 16..31; 2^s 12..15; pack P 8..15
      //   4: value-projection MFMAs and the X refills
      // The value MFMAs of the last tile follow the loop.
      constexpr int KPT = (KSC + NT - 1) / NT;  // hook k-steps per tile (at most)
      auto tl_of = [&](int n) __attribute__((always_inline)) { return tiles + (buf * W + n / NQW) * TILE; };
      auto ld_k = [&](int n, F (&kf)[KS]) __attribute__((always_inline)) {
#pragma unroll
        for (int js = 0; js < KS; ++js) kf[js] = load_frag(tl_of(n) + (hh * KS + js) * kFrag + lane * 8);
      };
      auto ld_v = [&](int n, F (&vf)[2][RB]) __attribute__((always_inline)) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            vf[hf][rb] = load_frag(tl_of(n) + (KFR + (hh * RB + rb) * 2 + hf) * kFrag + lane * 8);
      };
      auto ld_w = [&](int n, F (&wk)[KPT][GB], F (&wv)[KPT][GB]) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < KPT; ++q) {
          const int ks = n * KSC / NT + q;
          if (ks < (n + 1) * KSC / NT) {
#pragma unroll
            for (int cb = 0; cb < GB; ++cb) {
              const int fo = ((cb * KSC + ks) * 64 + lane) * 8;
              wk[q][cb] = load_frag(wk_l + fo);
              wv[q][cb] = load_frag(wv_l + fo);
            }
          }
        }
      };
      auto score_mma = [&](int n, const F (&kf)[KS]) __attribute__((always_inline)) {
        f32x16 sc;
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
        for (int js = 0; js < KS; ++js) mma(sc, kf[js], qf[n % NQW][js]);
        return sc;
      };
      F kc[KS], kn[KS], vc[2][RB], vn[2][RB], wkc[KPT][GB], wvc[KPT][GB], wkn[KPT][GB], wvn[KPT][GB];
      F pp[2], vp[2][RB];  // P and value operands of the previous tile
      ld_k(0, kc);
      ld_v(0, vc);
      ld_w(0, wkc, wvc);
      f32x16 cur = score_mma(0, kc);
      if (NT > 1) ld_k(1, kn);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int i = n % NQW, ip = (n + NQW - 1) % NQW;
        f32x16 nxt;
        // phase 0
        __builtin_amdgcn_sched_barrier(0);
        if (n + 1 < NT) {
          nxt = score_mma(n + 1, kn);
          ld_v(n + 1, vn);
          ld_w(n + 1, wkn, wvn);
          if (n + 2 < NT) {
            if ((n + 2) % NQW == 0) ld_k(n + 2, kc);  // kc is free: sub-tile of n + 2
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) cur[e] = __builtin_amdgcn_exp2f(cur[e]);
        // phase 1
        __builtin_amdgcn_sched_barrier(0);
        if (n > 0) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) mma(acc[ip][rb], vp[0][rb], pp[0]);
        }
#pragma unroll
        for (int e = 4; e < 8; ++e) cur[e] = __builtin_amdgcn_exp2f(cur[e]);
        F p0;
#pragma unroll
        for (int e = 0; e < 8; ++e) p0[e] = from_f32<T>(cur[e]);
        // phase 2
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < KPT; ++q) {
          const int ks = n * KSC / NT + q;
          if (ks < (n + 1) * KSC / NT) {
#pragma unroll
            for (int cb = 0; cb < GB; ++cb) mma(ka[cb], wkc[q][cb], xf[ks]);
          }
        }
#pragma unroll
        for (int e = 8; e < 12; ++e) cur[e] = __builtin_amdgcn_exp2f(cur[e]);
        if (!ONES_ROW) {
#pragma unroll
          for (int e = 0; e < 8; ++e) ls[i] += cur[e];
        }
        // phase 3
        __builtin_amdgcn_sched_barrier(0);
        if (n > 0) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) mma(acc[ip][rb], vp[1][rb], pp[1]);
        }
#pragma unroll
        for (int e = 12; e < 16; ++e) cur[e] = __builtin_amdgcn_exp2f(cur[e]);
        F p1;
#pragma unroll
        for (int e = 0; e < 8; ++e) p1[e] = from_f32<T>(cur[8 + e]);
        if (!ONES_ROW) {
#pragma unroll
          for (int e = 8; e < 16; ++e) ls[i] += cur[e];
        }
        // phase 4
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < KPT; ++q) {
          const int ks = n * KSC / NT + q;
          if (ks < (n + 1) * KSC / NT) {
#pragma unroll
            for (int cb = 0; cb < GB; ++cb) mma(va[cb], xf[ks], wvc[q][cb]);
            const int row = min(t0 + 2 * STEP + 32 * wave + c, k1 - 1);
            xf[ks] = load_frag(xb + (int64_t)row * p.C + 16 * ks + 8 * g);
          }
        }
        pp[0] = p0;
        pp[1] = p1;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) vp[hf][rb] = vc[hf][rb];
        if (n + 1 < NT) {
          cur = nxt;
#pragma unroll
          for (int hf = 0; hf < 2; ++hf)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) vc[hf][rb] = vn[hf][rb];
#pragma unroll
          for (int q = 0; q < KPT; ++q)
#pragma unroll
            for (int cb = 0; cb < GB; ++cb) { wkc[q][cb] = wkn[q][cb]; wvc[q][cb] = wvn[q][cb]; }
          if ((n + 2) % NQW == 0) {
#pragma unroll
            for (int js = 0; js < KS; ++js) kn[js] = kc[js];
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      {
        constexpr int il = (NT - 1) % NQW;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          mma(acc[il][rb], vp[0][rb], pp[0]);
          mma(acc[il][rb], vp[1][rb], pp[1]);
        }
      }
      return;
    }
    if constexpr (!MASK) {
      // Tiles n = j * NQW + i (sub-tile j, slot i); the score MFMA of tile
      // n + 1 is issued before the softmax of tile n, so its latency (and any
      // wait for the matrix pipe) is hidden behind the exponentials.
      F kfj[W][KS];
      auto score = [&](int n) __attribute__((always_inline)) {
        const int j = n / NQW, i = n % NQW;
        if (i == 0) {
          const T* tl = tiles + (buf * W + j) * TILE;
#pragma unroll
          for (int js = 0; js < KS; ++js) kfj[j][js] = load_frag(tl + (hh * KS + js) * kFrag + lane * 8);
        }
        f32x16 sc;
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
        for (int js = 0; js < KS; ++js) mma(sc, kfj[j][js], qf[i][js]);
        return sc;
      };
      f32x16 cur = score(0);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int j = n / NQW, i = n % NQW;
        f32x16 nxt;
        if (n + 1 < NT) nxt = score(n + 1);
        // keep the next score MFMA ahead of this tile's softmax
        __builtin_amdgcn_sched_barrier(0);
        const T* tl = tiles + (buf * W + j) * TILE;
        F vf[2][RB];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            vf[hf][rb] = load_frag(tl + (KFR + (hh * RB + rb) * 2 + hf) * kFrag + lane * 8);
        if (SF) tile_shift_free<T, RB, ONES_ROW, false>(acc[i], ls[i], cur, vf, 32, lane);
        else tile_online<T, RB, ONES_ROW, false>(acc[i], m[i], ls[i], cur, vf, 32, lane);
        hooks(n);
        if (n + 1 < NT) cur = nxt;
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < W; ++j) {
      int nvalid = 32;
      if (MASK) {
        nvalid = min(32, k1 - (t0 + 32 * j));
        if (nvalid <= 0) break;
      }
      const T* tl = tiles + (buf * W + j) * TILE;
      F kf[KS];
#pragma unroll
      for (int js = 0; js < KS; ++js) kf[js] = load_frag(tl + (hh * KS + js) * kFrag + lane * 8);
      F vf[2][RB];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          vf[hf][rb] = load_frag(tl + (KFR + (hh * RB + rb) * 2 + hf) * kFrag + lane * 8);
#pragma unroll
      for (int i = 0; i < NQW; ++i) {
        {
          f32x16 sc;
#pragma unroll
          for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
          for (int js = 0; js < KS; ++js) mma(sc, kf[js], qf[i][js]);
          if (SF) tile_shift_free<T, RB, ONES_ROW, MASK>(acc[i], ls[i], sc, vf, nvalid, lane);
          else tile_online<T, RB, ONES_ROW, MASK>(acc[i], m[i], ls[i], sc, vf, nvalid, lane);
        }
        hooks(j * NQW + i);
      }
    }
  };

  // Full super-tiles: shift-free while every score of the super-tile is
  // provably within the shift-free range (|q.k| <= max|q| max|k|), then
  // online from the first super-tile that fails the bound on; a partial last
  // super-tile runs online with masked keys.
  const int nfull = (k1 - k0) / STEP;
  const bool tail = (k1 - k0) % STEP != 0;
  const int nst = nfull + (tail ? 1 : 0);
  bool used = false;
  auto go_online = [&]() __attribute__((always_inline)) {
    if (!used) {
#pragma unroll
      for (int i = 0; i < NQW; ++i) m[i] = -INFINITY;
      used = true;
    }
  };
  // The shift-free super-tiles run in a loop of their own, so that its body
  // is a single path: with the shift-free and online bodies in one loop the
  // register allocator placed the loop-carried X rows differently in each
  // and copied them at every iteration, behind a wait for the X loads still
  // in flight.
  auto fast_at = [&](int it) __attribute__((always_inline)) {
    float kb = 0.f;
    for (int j = 0; j < W * HPG; ++j) kb = fmaxf(kb, kmx[(it & 1) * W * HPG + j]);
    return uniform(qmax2 * kb <= p.fast_lim);
  };
  auto next_super_tile = [&](int it) __attribute__((always_inline)) {
    if (it + 1 < nst) {  // the next super-tile, projected during this one
      proj_store((it + 1) & 1);
      lds_barrier();
    }
  };
  int t0 = k0, it = 0;
  if constexpr (!(D == 32 && KSC == 16)) {
    for (; it < nfull && fast_at(it); ++it, t0 += STEP) {
      consume(std::true_type{}, std::false_type{}, it, t0);
      used = true;
      next_super_tile(it);
    }
    if (it < nfull) go_online();
    for (; it < nfull; ++it, t0 += STEP) {
      consume(std::false_type{}, std::false_type{}, it, t0);
      next_super_tile(it);
    }
  } else {  // C = 256, D = 32: the two loops run out of registers; one loop
    bool fast = true;
    for (; it < nfull; ++it, t0 += STEP) {
      if (fast) fast = fast_at(it);
      if (fast) {
        consume(std::true_type{}, std::false_type{}, it, t0);
        used = true;
      } else {
        go_online();
        consume(std::false_type{}, std::false_type{}, it, t0);
      }
      next_super_tile(it);
    }
  }
  if (tail) {
    go_online();
    consume(std::false_type{}, std::true_type{}, nfull, t0);
  }

  // ---- partials ----
  // A chunk that starts at or past the last token holds no key: its partial
  // is (-inf, 0, 0) (App. A.3), whatever shift the loops above left in m.
  const bool empty_chunk = k1 <= k0;
  constexpr int NQ4 = ONES_ROW ? 2 : 4;
#pragma unroll
  for (int i = 0; i < NQW; ++i) {
    const int s = slot0 + i;
    if (s >= nslots) continue;
    if (empty_chunk) m[i] = -INFINITY;
    const int h = hg * HPG + hh, qb = s % p.QB;
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
// order, then the 16 slices of a row are folded pairwise (xor 1, 2, 4, 8);
// every slice then holds the whole row (equal up to the rounding order of its
// folds), and output element d is taken from slice d % 16.  Each thread issues the loads of kCombineBatch partials before folding any
// of them, so a batch costs one memory round trip.
// ---------------------------------------------------------------------------
constexpr int kCombineBatch = 4;

template <int D>
__device__ __forceinline__ void fold_partial(float& m, float& l, float (&a)[D], float mr, float lr,
                                             const float (&ar)[D]) {
  if (mr == -INFINITY) return;  // empty chunk: (-inf, 0, 0)
  const float mn = fmaxf(m, mr);
  const float wa = __builtin_amdgcn_exp2f(m - mn), wb = __builtin_amdgcn_exp2f(mr - mn);
  l = l * wa + lr * wb;
#pragma unroll
  for (int d = 0; d < D; ++d) a[d] = a[d] * wa + ar[d] * wb;
  m = mn;
}

template <typename T, int D>
__global__ __launch_bounds__(256) void k_combine_par(CombineParams p) {
  constexpr int KS = D / 16;
  const int t = threadIdx.x, rs = t & 15;
  // this thread's first preparation item: loads now, store at the end
  const int64_t pi0 = (int64_t)threadIdx.x * gridDim.x + blockIdx.x;
  typename Frag<T>::type pv;
  if (pi0 < p.prep_n) pv = prep_load<T>(p.prep, pi0);
  const int rows_per_bh = p.Mp / 16;
  const int64_t bh = blockIdx.x / rows_per_bh;
  const int qrow = (blockIdx.x % rows_per_bh) * 16 + (t >> 4);
  float m = -INFINITY, l = 0.f, a[D];
#pragma unroll
  for (int d = 0; d < D; ++d) a[d] = 0.f;
  for (int r0 = rs; r0 < p.R; r0 += 16 * kCombineBatch) {
    float mr[kCombineBatch], lr[kCombineBatch], ar[kCombineBatch][D];
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) {
      const int r = r0 + 16 * u;
      mr[u] = -INFINITY;
      lr[u] = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) ar[u][d] = 0.f;
      if (r < p.R) {
        const int64_t pidx = (bh * p.R + r) * p.Mp + qrow;
        const f32x2 ml = *reinterpret_cast<const f32x2*>(p.part_ml + pidx * 2);
        mr[u] = ml[0];
        lr[u] = ml[1];
#pragma unroll
        for (int d = 0; d < D; d += 4) {
          const f32x4 v = *reinterpret_cast<const f32x4*>(p.part_acc + pidx * D + d);
          ar[u][d] = v[0]; ar[u][d + 1] = v[1]; ar[u][d + 2] = v[2]; ar[u][d + 3] = v[3];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) fold_partial<D>(m, l, a, mr[u], lr[u], ar[u]);
  }
#pragma unroll
  for (int k = 1; k < 16; k <<= 1) {
    float ao[D];
#pragma unroll
    for (int d = 0; d < D; ++d) ao[d] = __shfl_xor(a[d], k, 64);
    const float mo = __shfl_xor(m, k, 64), lo = __shfl_xor(l, k, 64);
    fold_partial<D>(m, l, a, mo, lo, ao);
  }
  const bool valid = qrow < p.M;
  const float inv = (valid && l > 0.f) ? 1.f / l : 0.f;
  const int qb = qrow >> 5, qc = qrow & 31;
  if (p.frag && p.q_op && p.qnorm2) {
    // max over the wave's 4 rows of |scaled q|^2 (of the rounded operand),
    // one entry per wave
    float n2 = 0.f;
    if (valid) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const float q = to_f32(from_f32<T>(a[d] * inv * p.qscale));
        n2 = __builtin_fmaf(q, q, n2);
      }
    }
    n2 = fmaxf(n2, __shfl_xor(n2, 16, 64));
    n2 = fmaxf(n2, __shfl_xor(n2, 32, 64));
    if ((t & 63) == 0) p.qnorm2[bh * (p.Mp / 4) + (blockIdx.x % rows_per_bh) * 4 + (t >> 6)] = n2;
  }
#pragma unroll
  for (int d0 = 0; d0 < D; d0 += 16) {
    const int d = d0 + rs;
    float v = 0.f;
#pragma unroll
    for (int k = 0; k < D; ++k)
      if (k == d) v = a[k];
    const float out = v * inv;
    if (valid && p.out32) p.out32[(bh * p.M + qrow) * D + d] = out;
    if (p.q_rows) ((T*)p.q_rows)[(bh * p.Mp + qrow) * D + d] = from_f32<T>(out * p.qscale);
    if (p.z_rows) ((T*)p.z_rows)[(bh * D + d) * p.Mp + qrow] = from_f32<T>(out);
    if (!p.frag) {
      if (p.q_op) ((T*)p.q_op)[(bh * p.Mp + qrow) * D + d] = from_f32<T>(out * p.qscale);
      if (p.z_op) ((T*)p.z_op)[(bh * D + d) * p.Mp + qrow] = from_f32<T>(out);
    } else {
      if (p.q_op) {  // q fragment order
        const int js = d >> 4, gq = (d >> 3) & 1, jj = d & 7;
        const int64_t off = (int64_t)bh * p.Mp * D + ((int64_t)(qb * KS + js) * 64 + gq * 32 + qc) * 8 + jj;
        ((T*)p.q_op)[off] = from_f32<T>(out * p.qscale);
      }
      if (p.z_op) {  // z fragment order; row qc of route tile qb
        const int hf = qc >> 4, rr = qc & 15, gz = (rr >> 2) & 1, jj = 4 * (rr >> 3) + (rr & 3);
        T* z = (T*)p.z_op + bh * z_frag_elems_per_head(p.Mp, D);
        z[z_frag_index(qb, hf, d >> 5, gz, d & 31, jj, D)] = from_f32<T>(out);
      }
    }
  }
  if (valid && p.lse && rs == 0) p.lse[bh * p.M + qrow] = 0.6931471805599453f * (m + __log2f(l));
  if (pi0 < p.prep_n) prep_store<T>(p.prep, pi0, pv);
  for (int64_t k = 1;; ++k) {  // further items (when there are more than threads)
    const int64_t i = (k * blockDim.x + threadIdx.x) * gridDim.x + blockIdx.x;
    if (i >= p.prep_n) break;
    prep_store<T>(p.prep, i, prep_load<T>(p.prep, i));
  }
}

// Route tiles of the HPG heads of a group, software pipelined over the
// sequence (rt, hh): the score tile of the next pair is issued (its MFMA runs
// in the matrix pipe) before the softmax and value product of the current
// one.  score(rt, hh) returns a score tile, finish(rt, hh, s, mask) consumes
// it.  Route tiles below rt_full are whole; tile rt_full (when rt_full < RT)
// is the partial, masked one.
template <int HPG, class Score, class Finish>
__device__ __forceinline__ void pipelined_routes2(int RT, int rt_full, Score&& score, Finish&& finish) {
  f32x16 a = score(0, 0), bb;
  if constexpr (HPG == 2) {
    int rt = 0;
    for (; rt < rt_full; ++rt) {
      bb = score(rt, 1);
      finish(rt, 0, a, std::false_type{});
      if (rt + 1 < RT) a = score(rt + 1, 0);
      finish(rt, 1, bb, std::false_type{});
    }
    if (rt < RT) {
      bb = score(rt, 1);
      finish(rt, 0, a, std::true_type{});
      finish(rt, 1, bb, std::true_type{});
    }
  } else {
    int rt = 0;
    for (; rt + 2 <= rt_full; rt += 2) {
      bb = score(rt + 1, 0);
      finish(rt, 0, a, std::false_type{});
      if (rt + 2 < RT) a = score(rt + 2, 0);
      finish(rt + 1, 0, bb, std::false_type{});
    }
    if (rt < rt_full) {  // one whole tile left (scores in a), maybe a partial one after it
      const bool part = rt + 1 < RT;
      if (part) bb = score(rt + 1, 0);
      finish(rt, 0, a, std::false_type{});
      if (part) finish(rt + 1, 0, bb, std::true_type{});
    } else if (rt < RT) {  // only the partial tile left (scores in a)
      finish(rt, 0, a, std::true_type{});
    }
  }
}

// ---------------------------------------------------------------------------
// Decode with the key projection and the merge fused (call 3 + W_O).
// ---------------------------------------------------------------------------
// Waves (of 32 tokens) per decode workgroup: 8, two per SIMD (at C = 256 the
// resident X and Y fragments take 128 of each wave's 256 registers).
constexpr int dec_waves(int) { return 8; }

int decode_stage_elems(int C, int D, int Mp) {
  const int hpg = D == 16 ? 2 : 1, gb = D == 64 ? 2 : 1;
  const int head_stage = gb * (C / 16) * kFrag + hpg * (Mp * D + (int)z_frag_elems_per_head(Mp, D));
  const int wo_stage = (C / 16) * kFrag;
  return head_stage > wo_stage ? head_stage : wo_stage;
}

bool decode_fused_fits(int C, int D, int Mp, int elem_bytes) {
  return decode_kind_fits(decode_kind(C, D, Mp, elem_bytes), C, D, Mp, elem_bytes);
}

// Issue the global -> LDS copy of decode stage s into buffer s & 1: for
// s < HG [key weight slice][q fragments of the group's heads][z fragments of
// them]; for s = HG + cb the W_O fragments of output block cb.
template <typename T, int D, int KSC>
__device__ __forceinline__ void decode_stage_issue(const DecFusedParams& p, char* smem, int SE, int b, int s) {
  constexpr int HPG = (D == 16) ? 2 : 1, GB = (D == 64) ? 2 : 1;
  constexpr int C = KSC * 16, HG = C / 32 / GB, WELEMS = GB * KSC * kFrag;
  constexpr int NT = 64 * dec_waves(C), per16 = 16 / (int)sizeof(T);
  char* dst = smem + (size_t)(s & 1) * SE * sizeof(T);
  if (s >= HG) {
    copy_to_lds((const T*)p.wof + (int64_t)(s - HG) * KSC * kFrag, dst, KSC * kFrag / per16, NT);
    return;
  }
  const int64_t h0 = (int64_t)b * p.H + (int64_t)s * HPG;
  const int nq = HPG * p.Mp * D;
  const int64_t nz = (int64_t)HPG * z_frag_elems_per_head(p.Mp, D);
  copy_to_lds((const T*)p.wkf + (int64_t)s * WELEMS, dst, WELEMS / per16, NT);
  copy_to_lds((const T*)p.q_op + h0 * p.Mp * D, dst + (size_t)WELEMS * sizeof(T), nq / per16, NT);
  copy_to_lds((const T*)p.z_op + h0 * z_frag_elems_per_head(p.Mp, D), dst + (size_t)(WELEMS + nq) * sizeof(T),
              (int)(nz / per16), NT);
}

template <typename T, int D, int KSC>
__global__ __launch_bounds__(64 * dec_waves(16 * KSC)) void k_decode_fused(DecFusedParams p) {
  using F = typename Frag<T>::type;
  constexpr int HPG = (D == 16) ? 2 : 1, GB = (D == 64) ? 2 : 1;
  constexpr int KS = D / 16, RB = (D + 31) / 32;
  constexpr bool ONES_ROW = (D == 16);
  constexpr int C = KSC * 16, CB = C / 32, HG = CB / GB, H = C / D;
  constexpr int WELEMS = GB * KSC * kFrag;  // key weight slice of one head group
  constexpr int NW = dec_waves(C), TOK = 32 * NW;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  T* bufs = reinterpret_cast<T*>(smem);
  const int SE = p.stage_elems;

  const int lane = lane_id(), g = lane >> 5, c = lane & 31, wave = wave_id();
  const int nblk = (p.N + TOK - 1) / TOK;
  const int b = blockIdx.x / nblk;
  const int xrow = (blockIdx.x % nblk) * TOK + wave * 32 + c;
  const bool xok = xrow < p.N;
  const int Mp = p.Mp, RT = Mp / 32;
  const int ZH = (int)z_frag_elems_per_head(Mp, D);
  constexpr int ZC = D < 32 ? D : 32;  // value rows per z fragment
  // constant value-operand rows for D = 16 (after the two stage buffers):
  // 8 ones (row 16, the denominators), then 8 zeros (rows 17 .. 31)
  const int zconst_off = 2 * SE * (int)sizeof(T);
  if (ONES_ROW && threadIdx.x < 2)
    store_frag<T>(reinterpret_cast<T*>(smem + zconst_off) + 8 * threadIdx.x,
                  threadIdx.x == 0 ? fill_frag<T>(1.f) : zero_frag<T>());

  decode_stage_issue<T, D, KSC>(p, smem, SE, b, 0);
  F xf[KSC];
#pragma unroll
  for (int ks = 0; ks < KSC; ++ks)
    xf[ks] = load_frag((const T*)p.x + ((int64_t)b * p.N + min(xrow, p.N - 1)) * C + 16 * ks + 8 * g);
  // Route-query norm bound of every head (max over its routes of |scaled
  // q|^2, from the combine's per-wave entries), loaded once here behind
  // stage 0 and X.  A load issued inside the group loop is consumed at once,
  // and with in-order completion that wait would drain the stage copy issued
  // just before it.  Head h's bound ends up in lane h of qtab.
  int qtab = 0;
  {
    float qv[H];
#pragma unroll
    for (int h = 0; h < H; ++h) qv[h] = 0.f;
    for (int i = lane; i < Mp / 4; i += 64) {
      float t[H];
#pragma unroll
      for (int h = 0; h < H; ++h) t[h] = p.qnorm2[((int64_t)b * p.H + h) * (Mp / 4) + i];
#pragma unroll
      for (int h = 0; h < H; ++h) qv[h] = fmaxf(qv[h], t[h]);
    }
    lds_wait_barrier();
#pragma unroll
    for (int h = 0; h < H; ++h) qtab = lane == h ? __float_as_int(wave_max_nonneg(qv[h])) : qtab;
  }

  F yf[KSC];  // decoded tokens, merge B operands (16 channels per k step)
#pragma unroll
  for (int hg = 0; hg < HG; ++hg) {
    decode_stage_issue<T, D, KSC>(p, smem, SE, b, hg + 1);
    const T* sb = bufs + (hg & 1) * SE;
    f32x16 ka[GB];
#pragma unroll
    for (int cb = 0; cb < GB; ++cb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) ka[cb][e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KSC; ++ks) mma(ka[cb], load_frag(sb + ((cb * KSC + ks) * 64 + lane) * 8), xf[ks]);
    }
    // token keys of the group's heads, and the |score| bound (token-key
    // norms x the route-query norm bound); the heads of a group go through
    // one route loop together, shift-free only if both bounds allow it
    F kf[HPG][KS];
    float bnd = 0.f;
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
#pragma unroll
      for (int js = 0; js < KS; ++js) {
        const int fi = hh * KS + js;
        kf[hh][js] = cvt8<T>(ka[fi >> 1], 8 * (fi & 1));
      }
      bnd = fmaxf(bnd, frag_rows_max_sq<T, KS>(kf[hh]) *
                           __int_as_float(__builtin_amdgcn_readlane(qtab, hg * HPG + hh)));
    }
    const bool fast = uniform(bnd <= p.fast_lim);
    // z operand addresses (bytes into LDS): lanes of value rows walk the
    // head's z fragments; on D = 16 the lanes of rows 16 .. 31 read the
    // constant ones / zeros block instead
    const char* sbc = reinterpret_cast<const char*>(sb);
    uint32_t zbase[HPG], zstep;
    {
      const bool konst = ONES_ROW && c >= 16;
      zstep = konst ? 0u : (uint32_t)(2 * ZC * 8 * sizeof(T));
#pragma unroll
      for (int hh = 0; hh < HPG; ++hh)
        zbase[hh] = konst ? (uint32_t)(zconst_off + (c == 16 ? 0 : 8 * (int)sizeof(T)))
                          : (uint32_t)((sbc - smem) + (WELEMS + HPG * Mp * D + hh * ZH + (g * ZC + c) * 8) * sizeof(T));
    }
    f32x16 acc[HPG][RB];
    float m[HPG], ls[HPG];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      m[hh] = -INFINITY;
      ls[hh] = 0.f;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[hh][rb][e] = 0.f;
    }
    // all route tiles shift-free (sf = true) or online; only the last route
    // tile can be partial (M % 32 != 0) and it alone is masked
    const int rt_full = p.M / 32;
    auto score = [&](int rt, int hh) __attribute__((always_inline)) {
      f32x16 sc;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
      for (int js = 0; js < KS; ++js)
        mma(sc, load_frag(sb + WELEMS + hh * Mp * D + ((rt * KS + js) * 64 + lane) * 8), kf[hh][js]);
      return sc;
    };
    auto routes = [&](auto sf) __attribute__((always_inline)) {
      constexpr bool SF = decltype(sf)::value;
      auto finish = [&](int rt, int hh, const f32x16& sc, auto mask) __attribute__((always_inline)) {
        constexpr bool MASK = decltype(mask)::value;
        const int nvalid = MASK ? p.M - rt * 32 : 32;
        F zv[2][RB];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            zv[hf][rb] = *reinterpret_cast<const F*>(smem + zbase[hh] + zstep * ((rt * 2 + hf) * RB + rb));
        if (SF) tile_shift_free<T, RB, ONES_ROW, MASK>(acc[hh], ls[hh], sc, zv, nvalid, lane);
        else tile_online<T, RB, ONES_ROW, MASK>(acc[hh], m[hh], ls[hh], sc, zv, nvalid, lane);
      };
      if constexpr (KSC >= 16) {
        // C = 256: one score tile in flight (the software-pipelined order's
        // second tile would push the X and Y fragments out of registers)
        for (int rt = 0; rt < rt_full; ++rt)
#pragma unroll
          for (int hh = 0; hh < HPG; ++hh) finish(rt, hh, score(rt, hh), std::false_type{});
        if (rt_full < RT)
#pragma unroll
          for (int hh = 0; hh < HPG; ++hh) finish(rt_full, hh, score(rt_full, hh), std::true_type{});
      } else {
        pipelined_routes2<HPG>(RT, rt_full, score, finish);
      }
    };
    if (fast) routes(std::true_type{});
    else routes(std::false_type{});
    // the decoded tokens of the finished groups, oldest first: a shift
    // register, so that every index is a compile-time constant (the group
    // loop is not unrolled) and yf stays in registers
    constexpr int GKS = HPG * KS;  // fragments per group
#pragma unroll
    for (int u = 0; u + GKS < KSC; ++u) yf[u] = yf[u + GKS];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      const int h = hg * HPG + hh;
      const float den = softmax_denominator<RB, ONES_ROW>(acc[hh], ls[hh], lane);
      const float inv = __builtin_amdgcn_rcpf(den);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
          if (rb * 32 + 16 * hf < D) yf[KSC - GKS + hh * KS + 2 * rb + hf] = cvt8<T>(acc[hh][rb], 8 * hf, inv);
      // log2 of the softmax normaliser over the routes (0 is the shift of the
      // shift-free tiles), for the backward
      if (p.lse2 && xok && g == 0) p.lse2[((int64_t)b * H + (h)) * p.N + xrow] = (fast ? 0.f : m[hh]) + __log2f(den);
      if (p.y && xok) {
        T* yp = (T*)p.y + ((int64_t)b * p.N + xrow) * C + h * D;
        constexpr int NQ4 = ONES_ROW ? 2 : 4;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int q = 0; q < NQ4; ++q)
            store4(yp + rb * 32 + 8 * q + 4 * g, acc[hh][rb][4 * q] * inv, acc[hh][rb][4 * q + 1] * inv,
                   acc[hh][rb][4 * q + 2] * inv, acc[hh][rb][4 * q + 3] * inv);
      }
    }
    lds_wait_barrier();
  }

  // ---- merge: O^T = W_O^T Y^T, one 32-channel output block per stage ----
  // A block's stores are issued after the next barrier, and its residual is
  // loaded before its stage's copy: the barrier's wait for the next stage's
  // copy then covers both instead of draining the copy at each use.
  using Half = typename Frag<T>::half;
  auto load_res = [&](int cbo, Half (&r)[4]) __attribute__((always_inline)) {
    if (p.res && xok) {
      const T* rp = (const T*)p.res + ((int64_t)b * p.N + xrow) * C + 32 * cbo;
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = load_half(rp + 8 * q + 4 * g);
    }
  };
  auto store_o = [&](int cbo, const f32x16& o, const Half (&r)[4]) __attribute__((always_inline)) {
    if (xok) {
      T* op = (T*)p.o + ((int64_t)b * p.N + xrow) * C + 32 * cbo;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v[4] = {o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]};
        if (p.res) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += to_f32(r[q][e]);
        }
        store4(op + 8 * q + 4 * g, v[0], v[1], v[2], v[3]);
      }
    }
  };
  f32x16 o_prev;
  Half r_prev[4], r_cur[4];
#pragma unroll
  for (int cbo = 0; cbo < CB; ++cbo) {
    const int s = HG + cbo;
    if (cbo > 0) store_o(cbo - 1, o_prev, r_prev);
    load_res(cbo, r_cur);
    if (cbo + 1 < CB) decode_stage_issue<T, D, KSC>(p, smem, SE, b, s + 1);
    const T* sb = bufs + (s & 1) * SE;
    f32x16 o;
#pragma unroll
    for (int e = 0; e < 16; ++e) o[e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KSC; ++ks) mma(o, load_frag(sb + (ks * 64 + lane) * 8), yf[ks]);
    if (cbo + 1 < CB) lds_wait_barrier();
    o_prev = o;
#pragma unroll
    for (int q = 0; q < 4; ++q) r_prev[q] = r_cur[q];
  }
  store_o(CB - 1, o_prev, r_prev);
}

// ---------------------------------------------------------------------------
// Decode for C <= 128, one stage per head group.  A stage holds everything
// the group needs: [key weight slice][W_O rows of the group's channels (all
// output blocks)][q of its heads][z of its heads][route norm bounds].  With
// RES every stage is copied into LDS once at the start (when all fit) and the
// waves never synchronise again; otherwise two stage buffers alternate.  The
// merge accumulates O^T += W_O^T Y^T over the head groups, so the decoded
// tokens of a group are used as soon as they exist.
// ---------------------------------------------------------------------------
size_t dec2_stage_bytes(int C, int D, int Mp, int elem_bytes) {
  const int hpg = D == 16 ? 2 : 1, gb = D == 64 ? 2 : 1;
  const size_t el = (size_t)gb * (C / 16) * kFrag + (size_t)(C / 32) * 2 * gb * kFrag +
                    (size_t)hpg * ((size_t)Mp * D + z_frag_elems_per_head(Mp, D));
  return el * elem_bytes + (size_t)hpg * Mp;  // + hpg * Mp / 4 float bounds
}

size_t dec2_lds_bytes(int C, int D, int Mp, int elem_bytes, bool res) {
  const int hg = C / 32 / (D == 64 ? 2 : 1);
  return (res ? hg : 2) * dec2_stage_bytes(C, D, Mp, elem_bytes) + 16 * elem_bytes;
}

// LDS of k_decode_persist: [2 head stages][W_K fragments][W_O fragments]
// [16 constant elements]; a head stage is [q][z].  The kernel declares the
// whole 160 KB statically (one workgroup per CU in any case): a static array
// has a known address, so the route loop's LDS addresses need no add of the
// dynamic-LDS base, and the stages, first, are reached with the 16-bit
// immediate offsets of the LDS reads.
size_t persist_stage_bytes(int D, int Mp, int elem_bytes) {
  return (size_t)2 * Mp * D * elem_bytes;
}
size_t persist_lds_bytes(int C, int D, int Mp, int elem_bytes) {
  return (size_t)2 * C * C * elem_bytes + 2 * persist_stage_bytes(D, Mp, elem_bytes) + 16 * elem_bytes;
}

bool decode_kind_fits(int kind, int C, int D, int Mp, int elem_bytes) {
  switch (kind) {
    case kDecodeGroupsResident: return C <= 128 && dec2_lds_bytes(C, D, Mp, elem_bytes, true) <= 160 * 1024;
    case kDecodeGroupsStaged: return C <= 128 && dec2_lds_bytes(C, D, Mp, elem_bytes, false) <= 160 * 1024;
    case kDecodePersist:
      return elem_bytes == 2 && C <= 128 && (D == 16 || D == 32) && persist_lds_bytes(C, D, Mp, elem_bytes) <= kPersistLdsBytes;
    case kDecodeStaged: {
      const size_t se = (size_t)decode_stage_elems(C, D, Mp) * elem_bytes;
      return 2 * se + 16 * elem_bytes <= 160 * 1024;
    }
  }
  return false;
}

// Every route stage resident when it fits (k_decode3 / k_decode2), else the
// persistent decode with per-head stages, else the staged kernels.
int decode_kind(int C, int D, int Mp, int elem_bytes) {
  if (decode_kind_fits(kDecodeGroupsResident, C, D, Mp, elem_bytes)) return kDecodeGroupsResident;
  if (decode_kind_fits(kDecodePersist, C, D, Mp, elem_bytes)) return kDecodePersist;
  if (decode_kind_fits(kDecodeGroupsStaged, C, D, Mp, elem_bytes)) return kDecodeGroupsStaged;
  return kDecodeStaged;
}

template <typename T, int D, int KSC>
__device__ __forceinline__ void dec2_stage_issue(const DecFusedParams& p, char* dst, int b, int hg) {
  constexpr int HPG = (D == 16) ? 2 : 1, GB = (D == 64) ? 2 : 1;
  constexpr int C = KSC * 16, CB = C / 32, H = C / D, NT = 64 * dec_waves(C), PER16 = 16 / (int)sizeof(T);
  constexpr int WELEMS = GB * KSC * kFrag, WOE = CB * 2 * GB * kFrag;
  const int Mp = p.Mp, QE = HPG * Mp * D;
  const int ZE = HPG * (int)z_frag_elems_per_head(Mp, D);
  const int64_t h0 = (int64_t)b * H + hg * HPG;
  copy_to_lds((const T*)p.wkf + (int64_t)hg * WELEMS, dst, WELEMS / PER16, NT);
  dst += WELEMS * sizeof(T);
  copy_to_lds((const T*)p.wof + (int64_t)hg * WOE, dst, WOE / PER16, NT);
  dst += WOE * sizeof(T);
  copy_to_lds((const T*)p.q_op + h0 * Mp * D, dst, QE / PER16, NT);
  dst += QE * sizeof(T);
  copy_to_lds((const T*)p.z_op + h0 * z_frag_elems_per_head(Mp, D), dst, ZE / PER16, NT);
  dst += ZE * sizeof(T);
  copy_to_lds(p.qnorm2 + h0 * (Mp / 4), dst, HPG * Mp / 16, NT);
}

template <typename T, int D, int KSC, bool RES>
__global__ __launch_bounds__(64 * dec_waves(16 * KSC)) void k_decode2(DecFusedParams p) {
  using F = typename Frag<T>::type;
  constexpr int HPG = (D == 16) ? 2 : 1, GB = (D == 64) ? 2 : 1;
  constexpr int KS = D / 16, RB = (D + 31) / 32, KPG = 2 * GB;  // k steps (16 channels) per group
  constexpr bool ONES_ROW = (D == 16);
  constexpr int C = KSC * 16, CB = C / 32, HG = CB / GB;
  constexpr int WELEMS = GB * KSC * kFrag, WOE = CB * KPG * kFrag;
  constexpr int NW = dec_waves(C), TOK = 32 * NW;
  constexpr int ZC = D < 32 ? D : 32;  // value rows per z fragment
  static_assert(C <= 128, "per-group merge accumulators are sized for C <= 128");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int Mp = p.Mp, RT = Mp / 32, QH = Mp * D;
  const int ZH = (int)z_frag_elems_per_head(Mp, D);
  const int SB = p.stage_bytes;
  T* cst = reinterpret_cast<T*>(smem + (RES ? HG : 2) * SB);  // 8 ones (row 16), 8 zeros

  const int lane = lane_id(), g = lane >> 5, c = lane & 31, wave = wave_id();
  const int nblk = (p.N + TOK - 1) / TOK;
  const int b = blockIdx.x / nblk;
  const int xrow = (blockIdx.x % nblk) * TOK + wave * 32 + c;
  const bool xok = xrow < p.N;

  if (RES) {
    for (int hg = 0; hg < HG; ++hg) dec2_stage_issue<T, D, KSC>(p, smem + hg * SB, b, hg);
  } else {
    dec2_stage_issue<T, D, KSC>(p, smem, b, 0);
  }
  if (ONES_ROW && threadIdx.x < 2) store_frag<T>(cst + 8 * threadIdx.x, threadIdx.x == 0 ? fill_frag<T>(1.f) : zero_frag<T>());
  F xf[KSC];
#pragma unroll
  for (int ks = 0; ks < KSC; ++ks)
    xf[ks] = load_frag((const T*)p.x + ((int64_t)b * p.N + min(xrow, p.N - 1)) * C + 16 * ks + 8 * g);
  lds_wait_barrier();

  // z operand lanes: value-row lanes walk the head's z fragments; on D = 16
  // the lanes of rows 16 .. 31 read the constant block
  const bool konst = ONES_ROW && c >= 16;
  const uint32_t zstep = konst ? 0u : (uint32_t)(2 * ZC * 8 * sizeof(T));
  const uint32_t zhead = konst ? 0u : (uint32_t)(ZH * sizeof(T));
  const uint32_t zlane = konst ? (uint32_t)((reinterpret_cast<char*>(cst) - smem) + (c == 16 ? 0 : 8 * sizeof(T)))
                               : (uint32_t)((WELEMS + WOE + HPG * QH + (g * ZC + c) * 8) * sizeof(T));

  f32x16 o[CB];  // O^T blocks of this wave's 32 tokens
#pragma unroll
  for (int cb = 0; cb < CB; ++cb)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[cb][e] = 0.f;

  // key projection of head group hg from the stage at byte offset so
  auto project = [&](int so, f32x16 (&ka)[GB]) __attribute__((always_inline)) {
    const T* wk = reinterpret_cast<const T*>(smem + so);
#pragma unroll
    for (int cb = 0; cb < GB; ++cb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) ka[cb][e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KSC; ++ks) mma(ka[cb], load_frag(wk + ((cb * KSC + ks) * 64 + lane) * 8), xf[ks]);
    }
  };
  // max over a head's routes of |scaled q|^2 (wave-uniform), from its stage
  auto route_norm = [&](int so, int hh) __attribute__((always_inline)) {
    const float* qn = reinterpret_cast<const float*>(smem + so + (WELEMS + WOE + HPG * (QH + ZH)) * sizeof(T));
    float v = 0.f;
    for (int i = lane; i < Mp / 4; i += 64) v = fmaxf(v, qn[hh * (Mp / 4) + i]);
    return wave_max_nonneg(v);
  };
  // With every stage resident the next group's projection is issued before
  // this group's routes (the MFMAs run beside the softmax), and all route
  // norms are reduced up front.
  f32x16 ka[GB];
  float qn_all[RES ? HG * HPG : 1];
  if constexpr (RES) {
    project(0, ka);
#pragma unroll
    for (int i = 0; i < HG * HPG; ++i) qn_all[i] = route_norm((i / HPG) * SB, i % HPG);
  }

  for (int hg = 0; hg < HG; ++hg) {
    if (!RES && hg + 1 < HG) dec2_stage_issue<T, D, KSC>(p, smem + ((hg + 1) & 1) * SB, b, hg + 1);
    const int so = (RES ? hg : (hg & 1)) * SB;  // this group's stage (bytes)
    const T* st = reinterpret_cast<const T*>(smem + so);
    if constexpr (!RES) project(so, ka);
    // token keys of the group's heads
    F kf[HPG][KS];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh)
#pragma unroll
      for (int js = 0; js < KS; ++js) {
        const int fi = hh * KS + js;
        kf[hh][js] = cvt8<T>(ka[fi >> 1], 8 * (fi & 1));
      }
    // |score| bound: token-key norms x route-query norms; both heads of the
    // group go shift-free only if both bounds allow it
    float bnd = 0.f;
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      float qmax;
      if constexpr (RES) {
        qmax = 0.f;
#pragma unroll
        for (int i = 0; i < HG * HPG; ++i)
          if (i == hg * HPG + hh) qmax = qn_all[i];
      } else {
        qmax = route_norm(so, hh);
      }
      bnd = fmaxf(bnd, frag_rows_max_sq<T, KS>(kf[hh]) * qmax);
    }
    const bool fast = uniform(bnd <= p.fast_lim);
    if constexpr (RES) {
      if (hg + 1 < HG) project((hg + 1) * SB, ka);
    }

    f32x16 acc[HPG][RB];
    float m[HPG], ls[HPG];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      m[hh] = -INFINITY;
      ls[hh] = 0.f;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[hh][rb][e] = 0.f;
    }
    const int rt_full = p.M / 32;
    auto score = [&](int rt, int hh) __attribute__((always_inline)) {
      f32x16 sc;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
      for (int js = 0; js < KS; ++js)
        mma(sc, load_frag(st + WELEMS + WOE + hh * QH + ((rt * KS + js) * 64 + lane) * 8), kf[hh][js]);
      return sc;
    };
    auto zfrags = [&](int rt, int hh, F (&zv)[2][RB]) __attribute__((always_inline)) {
      const uint32_t base = zlane + (konst ? 0u : (uint32_t)so) + zhead * hh;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          zv[hf][rb] = *reinterpret_cast<const F*>(smem + base + zstep * ((rt * 2 + hf) * RB + rb));
    };
    if (fast) {
      auto finish = [&](int rt, int hh, const f32x16& sc, auto mask) __attribute__((always_inline)) {
        constexpr bool MASK = decltype(mask)::value;
        F zv[2][RB];
        zfrags(rt, hh, zv);
        tile_shift_free<T, RB, ONES_ROW, MASK>(acc[hh], ls[hh], sc, zv, MASK ? p.M - rt * 32 : 32, lane);
      };
      pipelined_routes2<HPG>(RT, rt_full, score, finish);
    } else {  // online maximum (rare): plain loop, every tile masked
      for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int hh = 0; hh < HPG; ++hh) {
          F zv[2][RB];
          zfrags(rt, hh, zv);
          tile_online<T, RB, ONES_ROW, true>(acc[hh], m[hh], ls[hh], score(rt, hh), zv, min(32, p.M - rt * 32), lane);
        }
      }
    }

    // decoded tokens of the group -> merge operands, and the partial merge
    F yg[KPG];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      const float den = softmax_denominator<RB, ONES_ROW>(acc[hh], ls[hh], lane);
      const float inv = __builtin_amdgcn_rcpf(den);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
          if (rb * 32 + 16 * hf < D) yg[hh * KS + 2 * rb + hf] = cvt8<T>(acc[hh][rb], 8 * hf, inv);
      // log2 of the softmax normaliser over the routes (0 is the shift of the
      // shift-free tiles), for the backward
      if (p.lse2 && xok && g == 0) p.lse2[((int64_t)b * p.H + (hg * HPG + hh)) * p.N + xrow] = (fast ? 0.f : m[hh]) + __log2f(den);
      if (p.y && xok) {
        T* yp = (T*)p.y + ((int64_t)b * p.N + xrow) * C + (hg * HPG + hh) * D;
        constexpr int NQ4 = ONES_ROW ? 2 : 4;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int q = 0; q < NQ4; ++q)
            store4(yp + rb * 32 + 8 * q + 4 * g, acc[hh][rb][4 * q] * inv, acc[hh][rb][4 * q + 1] * inv,
                   acc[hh][rb][4 * q + 2] * inv, acc[hh][rb][4 * q + 3] * inv);
      }
    }
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int j = 0; j < KPG; ++j) mma(o[cb], load_frag(st + WELEMS + ((cb * KPG + j) * 64 + lane) * 8), yg[j]);
    if (!RES && hg + 1 < HG) lds_wait_barrier();  // next stage in; this one free
  }

  if (xok) {
    const int64_t oo = ((int64_t)b * p.N + xrow) * C;
    Res16<T> res[CB];
    if (p.res) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) load_res16(res[cb], (const T*)p.res + oo + 32 * cb, g);
    }
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) store16((T*)p.o + oo + 32 * cb, o[cb], res[cb], p.res != nullptr, g);
  }
}

// ---------------------------------------------------------------------------
// Decode with every stage resident and a compile-time route-tile count RT.
// The route tiles of a group are unrolled and software pipelined as the
// encode's shift-free tiles, with the key projection of the next group spread
// over them.  The decoded tokens of every group are kept (as MFMA operands)
// and the merge O^T = W_O^T Y^T runs after the last group, one 32-channel
// output block at a time, so the merge accumulators never share the register
// budget with the route tiles.  Same LDS layout and stages as
// k_decode2<..., RES = true>.
// ---------------------------------------------------------------------------
template <typename T, int D, int KSC, int RT>
__global__ __launch_bounds__(64 * dec_waves(16 * KSC)) void k_decode3(DecFusedParams p) {
  using F = typename Frag<T>::type;
  constexpr int HPG = (D == 16) ? 2 : 1, GB = (D == 64) ? 2 : 1;
  constexpr int KS = D / 16, RB = (D + 31) / 32, KPG = 2 * GB;
  constexpr bool ONES_ROW = (D == 16);
  constexpr int C = KSC * 16, CB = C / 32, HG = CB / GB;
  constexpr int WELEMS = GB * KSC * kFrag, WOE = CB * KPG * kFrag;
  constexpr int NW = dec_waves(C), TOK = 32 * NW;
  constexpr int ZC = D < 32 ? D : 32;
  constexpr int NT = RT * HPG;      // route tiles per group
  constexpr int NP = GB * KSC;      // projection MFMAs per group
  static_assert(C <= 128, "the decoded tokens of every group are kept in registers");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int Mp = p.Mp, QH = Mp * D;
  const int ZH = (int)z_frag_elems_per_head(Mp, D);
  const int SB = p.stage_bytes;
  T* cst = reinterpret_cast<T*>(smem + HG * SB);

  const int lane = lane_id(), g = lane >> 5, c = lane & 31, wave = wave_id();
  const int nblk = (p.N + TOK - 1) / TOK;
  const int b = blockIdx.x / nblk;
  const int xrow = (blockIdx.x % nblk) * TOK + wave * 32 + c;
  const bool xok = xrow < p.N;

  // X and every stage at once (group hg also reads stage hg + 1: the key
  // weights of the next group's projection); one wait, and no barrier inside
  // the group loop, where the waves drift apart by up to a microsecond
  F xf[KSC];
#pragma unroll
  for (int ks = 0; ks < KSC; ++ks)
    xf[ks] = load_frag((const T*)p.x + ((int64_t)b * p.N + min(xrow, p.N - 1)) * C + 16 * ks + 8 * g);
#pragma unroll
  for (int s0 = 0; s0 < HG; ++s0) dec2_stage_issue<T, D, KSC>(p, smem + s0 * SB, b, s0);
  if (ONES_ROW && threadIdx.x < 2) store_frag<T>(cst + 8 * threadIdx.x, threadIdx.x == 0 ? fill_frag<T>(1.f) : zero_frag<T>());
  lds_wait_barrier();

  const bool konst = ONES_ROW && c >= 16;
  const uint32_t zstep = konst ? 0u : (uint32_t)(2 * ZC * 8 * sizeof(T));
  const uint32_t zhead = konst ? 0u : (uint32_t)(ZH * sizeof(T));
  const uint32_t zlane = konst ? (uint32_t)((reinterpret_cast<char*>(cst) - smem) + (c == 16 ? 0 : 8 * sizeof(T)))
                               : (uint32_t)((WELEMS + WOE + HPG * QH + (g * ZC + c) * 8) * sizeof(T));

  f32x16 ka[GB];
  // decoded tokens of the finished groups, oldest first (a shift register:
  // after the last group entry hg holds group hg)
  F yall[HG][KPG];
#pragma unroll
  for (int u = 0; u < HG; ++u)
#pragma unroll
    for (int j = 0; j < KPG; ++j) yall[u][j] = zero_frag<T>();
  // k-th projection MFMA of the group whose stage starts at byte `so`
  auto proj_mfma = [&](int so, int k) __attribute__((always_inline)) {
    const int cb = k / KSC, ks = k % KSC;
    const T* wk = reinterpret_cast<const T*>(smem + so);
    if (ks == 0) {
#pragma unroll
      for (int e = 0; e < 16; ++e) ka[cb][e] = 0.f;
    }
    mma(ka[cb], load_frag(wk + ((cb * KSC + ks) * 64 + lane) * 8), xf[ks]);
  };
  auto route_norm = [&](int so, int hh) __attribute__((always_inline)) {
    const float* qn = reinterpret_cast<const float*>(smem + so + (WELEMS + WOE + HPG * (QH + ZH)) * sizeof(T));
    float v = 0.f;
    for (int i = lane; i < Mp / 4; i += 64) v = fmaxf(v, qn[hh * (Mp / 4) + i]);
    return wave_max_nonneg(v);
  };
#pragma unroll
  for (int k = 0; k < NP; ++k) proj_mfma(0, k);

  const bool partial = p.M < 32 * RT;  // the last route tile is partial
  for (int hg = 0; hg < HG; ++hg) {
    const int so = hg * SB;
    const T* st = reinterpret_cast<const T*>(smem + so);
    F kf[HPG][KS];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh)
#pragma unroll
      for (int js = 0; js < KS; ++js) {
        const int fi = hh * KS + js;
        kf[hh][js] = cvt8<T>(ka[fi >> 1], 8 * (fi & 1));
      }
    // |score| bound for both heads of the group at once: max |k|^2 over the
    // group's heads times max |q|^2 over its routes
    float ksq = 0.f, qsq = 0.f;
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      float sq = 0.f;
#pragma unroll
      for (int js = 0; js < KS; ++js) sq += sumsq(kf[hh][js]);
      ksq = fmaxf(ksq, sq);
      qsq = fmaxf(qsq, route_norm(so, hh));
    }
    const bool fast = uniform(halfmax_sum_nonneg(ksq) * qsq <= p.fast_lim);
    // the next group's stage (the last group projects its own again: unused)
    const int so_next = min(hg + 1, HG - 1) * SB;

    f32x16 acc[HPG][RB];
    float m[HPG], ls[HPG];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      m[hh] = -INFINITY;
      ls[hh] = 0.f;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[hh][rb][e] = 0.f;
    }
    auto ld_q = [&](int n, F (&qv)[KS]) __attribute__((always_inline)) {
      const int rt = n / HPG, hh = n % HPG;
#pragma unroll
      for (int js = 0; js < KS; ++js)
        qv[js] = load_frag(st + WELEMS + WOE + hh * QH + ((rt * KS + js) * 64 + lane) * 8);
    };
    auto score_q = [&](int n, const F (&qv)[KS]) __attribute__((always_inline)) {
      const int hh = n % HPG;
      f32x16 sc;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
      for (int js = 0; js < KS; ++js) mma(sc, qv[js], kf[hh][js]);
      return sc;
    };
    auto score = [&](int n) __attribute__((always_inline)) {
      F qv[KS];
      ld_q(n, qv);
      return score_q(n, qv);
    };
    auto zfrags = [&](int n, F (&zv)[2][RB]) __attribute__((always_inline)) {
      const int rt = n / HPG, hh = n % HPG;
      const uint32_t base = zlane + (konst ? 0u : (uint32_t)so) + zhead * hh;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          zv[hf][rb] = *reinterpret_cast<const F*>(smem + base + zstep * ((rt * 2 + hf) * RB + rb));
    };
    // the next group's key projection, spread after the route tiles
    constexpr int PK = (NP + NT - 1) / NT;  // projection k-steps per tile (at most)
    auto hooks = [&](int n) __attribute__((always_inline)) {
#pragma unroll
      for (int k = n * NP / NT; k < (n + 1) * NP / NT; ++k) proj_mfma(so_next, k);
    };
    if (fast && !partial) {
      // Software pipelined as the encode's shift-free tiles.  Per tile n:
      //   0: LDS reads (route keys of tile n + 2, latents of tile n - 1,
      //      projection weights of tile n); 2^s of scores 0..3
      //   1: value MFMAs of tile n - 1, routes 0..15; 2^s 4..7; pack P 0..7
      //   2: projection MFMAs (next group); 2^s 8..11
      //   3: value MFMAs of tile n - 1, routes 16..31; 2^s 12..15; pack P 8..15
      //   4: score MFMA of tile n + 1 (into this tile's score registers)
      F qc[KS], qn[KS], zp[2][RB], pp[2], wp[PK];
      ld_q(0, qc);
      f32x16 cur = score_q(0, qc);
      if (NT > 1) ld_q(1, qn);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int hh = n % HPG, hp = (n + HPG - 1) % HPG;
        // phase 0
        __builtin_amdgcn_sched_barrier(0);
        if (n > 0) zfrags(n - 1, zp);
#pragma unroll
        for (int u = 0; u < PK; ++u) {
          const int k = n * NP / NT + u;
          if (k < (n + 1) * NP / NT) wp[u] = load_frag(reinterpret_cast<const T*>(smem + so_next) + (k * 64 + lane) * 8);
        }
        if (n + 2 < NT) ld_q(n + 2, qc);  // qc is free
#pragma unroll
        for (int e = 0; e < 4; ++e) cur[e] = __builtin_amdgcn_exp2f(cur[e]);
        // phase 1
        __builtin_amdgcn_sched_barrier(0);
        if (n > 0) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) mma(acc[hp][rb], zp[0][rb], pp[0]);
        }
#pragma unroll
        for (int e = 4; e < 8; ++e) cur[e] = __builtin_amdgcn_exp2f(cur[e]);
        F p0;
#pragma unroll
        for (int e = 0; e < 8; ++e) p0[e] = from_f32<T>(cur[e]);
        // phase 2
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < PK; ++u) {
          const int k = n * NP / NT + u;
          if (k < (n + 1) * NP / NT) {
            const int cb = k / KSC, ks = k % KSC;
            if (ks == 0) {
#pragma unroll
              for (int e = 0; e < 16; ++e) ka[cb][e] = 0.f;
            }
            mma(ka[cb], wp[u], xf[ks]);
          }
        }
#pragma unroll
        for (int e = 8; e < 12; ++e) cur[e] = __builtin_amdgcn_exp2f(cur[e]);
        if (!ONES_ROW) {
#pragma unroll
          for (int e = 0; e < 8; ++e) ls[hh] += cur[e];
        }
        // phase 3
        __builtin_amdgcn_sched_barrier(0);
        if (n > 0) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) mma(acc[hp][rb], zp[1][rb], pp[1]);
        }
#pragma unroll
        for (int e = 12; e < 16; ++e) cur[e] = __builtin_amdgcn_exp2f(cur[e]);
        F p1;
#pragma unroll
        for (int e = 0; e < 8; ++e) p1[e] = from_f32<T>(cur[8 + e]);
        if (!ONES_ROW) {
#pragma unroll
          for (int e = 8; e < 16; ++e) ls[hh] += cur[e];
        }
        // phase 4
        __builtin_amdgcn_sched_barrier(0);
        if (n + 1 < NT) cur = score_q(n + 1, qn);
        pp[0] = p0;
        pp[1] = p1;
        if (n + 1 < NT) {
#pragma unroll
          for (int js = 0; js < KS; ++js) qn[js] = qc[js];
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      zfrags(NT - 1, zp);
      {
        constexpr int hl = (NT - 1) % HPG;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          mma(acc[hl][rb], zp[0][rb], pp[0]);
          mma(acc[hl][rb], zp[1][rb], pp[1]);
        }
      }
    } else if (fast) {
      f32x16 cur = score(0);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        f32x16 nxt;
        if (n + 1 < NT) nxt = score(n + 1);
        // keep the next score MFMA ahead of this tile's softmax
        __builtin_amdgcn_sched_barrier(0);
        F zv[2][RB];
        zfrags(n, zv);
        const int rt = n / HPG, hh = n % HPG;
        if (rt == RT - 1 && partial)
          tile_shift_free<T, RB, ONES_ROW, true>(acc[hh], ls[hh], cur, zv, p.M - rt * 32, lane);
        else
          tile_shift_free<T, RB, ONES_ROW, false>(acc[hh], ls[hh], cur, zv, 32, lane);
        hooks(n);
        if (n + 1 < NT) cur = nxt;
      }
    } else {  // online maximum (rare): every tile masked, matrix work afterwards
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int rt = n / HPG, hh = n % HPG;
        F zv[2][RB];
        zfrags(n, zv);
        tile_online<T, RB, ONES_ROW, true>(acc[hh], m[hh], ls[hh], score(n), zv, min(32, p.M - rt * 32), lane);
      }
#pragma unroll
      for (int n = 0; n < NT; ++n) hooks(n);
    }
    // this group's decoded tokens join the merge operands
#pragma unroll
    for (int u = 0; u + 1 < HG; ++u)
#pragma unroll
      for (int j = 0; j < KPG; ++j) yall[u][j] = yall[u + 1][j];
#pragma unroll
    for (int hh = 0; hh < HPG; ++hh) {
      const float den = softmax_denominator<RB, ONES_ROW>(acc[hh], ls[hh], lane);
      const float inv = __builtin_amdgcn_rcpf(den);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
          if (rb * 32 + 16 * hf < D) yall[HG - 1][hh * KS + 2 * rb + hf] = cvt8<T>(acc[hh][rb], 8 * hf, inv);
      // log2 of the softmax normaliser over the routes (0 is the shift of the
      // shift-free tiles), for the backward
      if (p.lse2 && xok && g == 0) p.lse2[((int64_t)b * p.H + (hg * HPG + hh)) * p.N + xrow] = (fast ? 0.f : m[hh]) + __log2f(den);
      if (p.y && xok) {
        T* yp = (T*)p.y + ((int64_t)b * p.N + xrow) * C + (hg * HPG + hh) * D;
        constexpr int NQ4 = ONES_ROW ? 2 : 4;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int q = 0; q < NQ4; ++q)
            store4(yp + rb * 32 + 8 * q + 4 * g, acc[hh][rb][4 * q] * inv, acc[hh][rb][4 * q + 1] * inv,
                   acc[hh][rb][4 * q + 2] * inv, acc[hh][rb][4 * q + 3] * inv);
      }
    }
  }
  // merge: output block cb of O^T = sum over the groups of W_O^T rows x Y^T
  // (the residual of every block is loaded before the first MFMA)
  const int64_t oo = ((int64_t)b * p.N + xrow) * C;
  Res16<T> res[CB];
  if (p.res && xok) {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) load_res16(res[cb], (const T*)p.res + oo + 32 * cb, g);
  }
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    f32x16 oc;
#pragma unroll
    for (int e = 0; e < 16; ++e) oc[e] = 0.f;
#pragma unroll
    for (int u = 0; u < HG; ++u) {
      const T* wo = reinterpret_cast<const T*>(smem + u * SB) + WELEMS;
#pragma unroll
      for (int j = 0; j < KPG; ++j) mma(oc, load_frag(wo + ((cb * KPG + j) * 64 + lane) * 8), yall[u][j]);
    }
    if (xok) store16((T*)p.o + oo + 32 * cb, oc, res[cb], p.res != nullptr, g);
  }
}

// ---------------------------------------------------------------------------
// Persistent decode (call 3 + merge) for C <= 128 when the route operands of
// every head do not fit in LDS together.  One workgroup of 8 waves per CU
// walks token blocks of 256 (t = blockIdx.x, blockIdx.x + gridDim.x, ...).
// W_K and W_O stay resident in LDS for the whole launch; the route operands
// of one head at a time ([q][z][route-norm bounds], one batch entry's head)
// go through two alternating stages, so the stage sequence runs on across
// token blocks: while head h is routed, the copy of the next head (or of head
// 0 of the next token block) is in flight.  The route-norm bound of every head
// is reduced once per batch entry, from the combine's per-wave maxima.  The X rows of the next token
// block are loaded once the last head group has been projected.  Per token
// block: HG key projections, H route loops, one merge O^T = W_O^T Y^T from
// the resident W_O (no barrier), and one barrier per head.
// ---------------------------------------------------------------------------
template <typename T, int D, int KSC>
__device__ __forceinline__ void persist_stage_issue(const DecFusedParams& p, char* dst, int bh) {
  constexpr int NT = 64 * dec_waves(16 * KSC), PER16 = 16 / (int)sizeof(T);
  const int Mp = p.Mp;
  const int QE = Mp * D, ZE = (int)z_frag_elems_per_head(Mp, D);
  copy_to_lds((const T*)p.q_op + (int64_t)bh * QE, dst, QE / PER16, NT);
  copy_to_lds((const T*)p.z_op + (int64_t)bh * ZE, dst + (size_t)QE * sizeof(T), ZE / PER16, NT);
}

template <typename T, int D, int KSC>
__global__ __launch_bounds__(64 * dec_waves(16 * KSC)) void k_decode_persist(DecFusedParams p) {
  using F = typename Frag<T>::type;
  constexpr int HPG = (D == 16) ? 2 : 1, GB = (D == 64) ? 2 : 1;
  constexpr int KS = D / 16, RB = (D + 31) / 32, KPG = 2 * GB;
  constexpr bool ONES_ROW = (D == 16);
  constexpr int C = KSC * 16, CB = C / 32, HG = CB / GB, H = C / D;
  constexpr int WELEMS = GB * KSC * kFrag;  // key weight slice of one head group
  constexpr int NW = dec_waves(C), TOK = 32 * NW;
  constexpr int ZC = D < 32 ? D : 32;
  constexpr int GKS = HPG * KS;  // decoded-token fragments per head group
  static_assert(C <= 128 && GKS == KPG, "");
  __shared__ __attribute__((aligned(16))) char smem[kPersistLdsBytes];
  const int Mp = p.Mp, RT = Mp / 32, QE = Mp * D;
  const int SB = p.stage_bytes;  // the host keeps 2 SB bytes + (2 C^2 + 16) elements within the array
  char* stage0 = smem;
  T* wk_l = reinterpret_cast<T*>(smem + 2 * SB);
  T* wo_l = wk_l + C * C;
  T* cst = wo_l + C * C;  // 8 ones (row 16), 8 zeros

  const int lane = lane_id(), g = lane >> 5, c = lane & 31, wave = wave_id();
  const int nblk = (p.N + TOK - 1) / TOK;
  const int total = p.B * nblk;
  int t = blockIdx.x;
  if (t >= total) return;  // whole workgroup, before any barrier

  // resident weights, the first head's stage and the first block's X
  copy_to_lds(p.wkf, reinterpret_cast<char*>(wk_l), C * C * (int)sizeof(T) / 16, 64 * NW);
  copy_to_lds(p.wof, reinterpret_cast<char*>(wo_l), C * C * (int)sizeof(T) / 16, 64 * NW);
  persist_stage_issue<T, D, KSC>(p, stage0, (t / nblk) * H);
  if (ONES_ROW && threadIdx.x < 2) store_frag<T>(cst + 8 * threadIdx.x, threadIdx.x == 0 ? fill_frag<T>(1.f) : zero_frag<T>());
  F xf[KSC];
  auto load_x = [&](int tb) __attribute__((always_inline)) {
    const int bb = tb / nblk, row = min((tb % nblk) * TOK + wave * 32 + c, p.N - 1);
#pragma unroll
    for (int ks = 0; ks < KSC; ++ks) xf[ks] = load_frag((const T*)p.x + ((int64_t)bb * p.N + row) * C + 16 * ks + 8 * g);
  };
  load_x(t);
  lds_wait_barrier();  // the weights are read before the first head's barrier

  // z operand lanes: value-row lanes walk the head's z fragments; on D = 16
  // the lanes of rows 16 .. 31 read the constant block
  const bool konst = ONES_ROW && c >= 16;
  const uint32_t zstep = konst ? 0u : (uint32_t)(2 * ZC * 8 * sizeof(T));
  const uint32_t zlane = konst ? (uint32_t)((reinterpret_cast<char*>(cst) - smem) + (c == 16 ? 0 : 8 * sizeof(T)))
                               : (uint32_t)((stage0 - smem) + (QE + (g * ZC + c) * 8) * sizeof(T));
  const int rt_full = p.M / 32;

  int seq = 0;  // stages consumed by this workgroup (buffer seq & 1)
  int bq = -1;  // the batch entry whose route-norm bounds qmax holds
  float qmax[H];
  for (; t < total; t += gridDim.x) {
    const int b = t / nblk;
    if (b != bq) {  // max over a head's routes of |scaled q|^2, wave-uniform
#pragma unroll
      for (int h = 0; h < H; ++h) {
        const float* qn = p.qnorm2 + ((int64_t)b * H + h) * (Mp / 4);
        float v = 0.f;
        for (int i = lane; i < Mp / 4; i += 64) v = fmaxf(v, qn[i]);
        qmax[h] = wave_max_nonneg(v);
      }
      bq = b;
    }
    const int xrow = (t % nblk) * TOK + wave * 32 + c;
    const bool xok = xrow < p.N;
    const int tn = t + gridDim.x;  // the next token block of this workgroup
    F yf[KSC];                     // decoded tokens, oldest group first (shift register)
    bool xpending = false;         // the next block's X loads are in flight
    for (int hg = 0; hg < HG; ++hg) {
      // key projection of the group's heads from the resident W_K slice
      f32x16 ka[GB];
#pragma unroll
      for (int cb = 0; cb < GB; ++cb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) ka[cb][e] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KSC; ++ks)
          mma(ka[cb], load_frag(wk_l + hg * WELEMS + ((cb * KSC + ks) * 64 + lane) * 8), xf[ks]);
      }
      F kf[HPG][KS];
#pragma unroll
      for (int hh = 0; hh < HPG; ++hh)
#pragma unroll
        for (int js = 0; js < KS; ++js) {
          const int fi = hh * KS + js;
          kf[hh][js] = cvt8<T>(ka[fi >> 1], 8 * (fi & 1));
        }
#pragma unroll
      for (int u = 0; u + GKS < KSC; ++u) yf[u] = yf[u + GKS];
#pragma unroll
      for (int hh = 0; hh < HPG; ++hh) {
        const int h = hg * HPG + hh;
        // This head's stage has landed (every wave's share of the copy) and
        // every wave is done with the previous one, whose buffer takes the
        // next.  Only the KSC loads of the next block's X rows (issued after
        // the copy, see below) may stay in flight across the barrier.
        if (xpending) {
          asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(KSC) : "memory");
        } else {
          asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
        }
        const int buf = seq & 1;
        ++seq;
        if (h + 1 < H) persist_stage_issue<T, D, KSC>(p, stage0 + (buf ^ 1) * SB, b * H + h + 1);
        else if (tn < total) persist_stage_issue<T, D, KSC>(p, stage0 + (buf ^ 1) * SB, (tn / nblk) * H);
        // X is no longer needed once the last group is projected: the next
        // token block's rows are loaded behind the first copy issued after it
        if (hg == HG - 1 && hh == 0 && tn < total) {
          asm volatile("" ::: "memory");  // the loads stay behind the copy: vmcnt(KSC) covers it
          load_x(tn);
          xpending = true;
        }
        const char* st = stage0 + buf * SB;
        // |score| bound: token-key norms x the head's route-query norm bound
        // (h is wave-uniform: the selection runs on scalar registers)
        float qh = qmax[0];
#pragma unroll
        for (int i = 1; i < H; ++i) qh = (h == i) ? qmax[i] : qh;
        const bool fast = uniform(frag_rows_max_sq<T, KS>(kf[hh]) * qh <= p.fast_lim);
        const T* qst = reinterpret_cast<const T*>(st);
        const uint32_t zb = zlane + (konst ? 0u : (uint32_t)(buf * SB));
        f32x16 acc[RB];
        float m = -INFINITY, ls = 0.f;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[rb][e] = 0.f;
        auto score = [&](int rt, int) __attribute__((always_inline)) {
          f32x16 sc;
#pragma unroll
          for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
          for (int js = 0; js < KS; ++js) mma(sc, load_frag(qst + ((rt * KS + js) * 64 + lane) * 8), kf[hh][js]);
          return sc;
        };
        auto routes = [&](auto sf) __attribute__((always_inline)) {
          constexpr bool SF = decltype(sf)::value;
          auto finish = [&](int rt, int, const f32x16& sc, auto mask) __attribute__((always_inline)) {
            constexpr bool MASK = decltype(mask)::value;
            const int nvalid = MASK ? p.M - rt * 32 : 32;
            F zv[2][RB];
#pragma unroll
            for (int hf = 0; hf < 2; ++hf)
#pragma unroll
              for (int rb = 0; rb < RB; ++rb)
                zv[hf][rb] = *reinterpret_cast<const F*>(smem + zb + zstep * ((rt * 2 + hf) * RB + rb));
            if (SF) tile_shift_free<T, RB, ONES_ROW, MASK>(acc, ls, sc, zv, nvalid, lane);
            else tile_online<T, RB, ONES_ROW, MASK>(acc, m, ls, sc, zv, nvalid, lane);
          };
          pipelined_routes2<1>(RT, rt_full, score, finish);
        };
        if (fast) routes(std::true_type{});
        else routes(std::false_type{});
        const float den = softmax_denominator<RB, ONES_ROW>(acc, ls, lane);
        const float inv = __builtin_amdgcn_rcpf(den);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int hf = 0; hf < 2; ++hf)
            if (rb * 32 + 16 * hf < D) yf[KSC - GKS + hh * KS + 2 * rb + hf] = cvt8<T>(acc[rb], 8 * hf, inv);
        // log2 of the softmax normaliser over the routes (0 is the shift of the
        // shift-free tiles), for the backward
        if (p.lse2 && xok && g == 0) p.lse2[((int64_t)b * H + (h)) * p.N + xrow] = (fast ? 0.f : m) + __log2f(den);
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
    }
    // merge: output block cb of O^T = sum over the groups of W_O^T rows x Y^T
    // (the residual of every block is loaded before the first MFMA)
    const int64_t oo = ((int64_t)b * p.N + xrow) * C;
    Res16<T> res[CB];
    if (p.res && xok) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) load_res16(res[cb], (const T*)p.res + oo + 32 * cb, g);
    }
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      f32x16 oc;
#pragma unroll
      for (int e = 0; e < 16; ++e) oc[e] = 0.f;
#pragma unroll
      for (int u = 0; u < HG; ++u)
#pragma unroll
        for (int j = 0; j < KPG; ++j)
          mma(oc, load_frag(wo_l + (((u * CB + cb) * KPG + j) * 64 + lane) * 8), yf[u * KPG + j]);
      if (xok) store16((T*)p.o + oo + 32 * cb, oc, res[cb], p.res != nullptr, g);
    }
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T, int D, int KSC, int NQW, int W>
static hipError_t enc_one(const EncFusedParams& p, hipStream_t s) {
  if constexpr (NQW > enc_nqw_cap(D, W, (int)sizeof(T)) || (W == 8 && !((D == 16 && KSC <= 8) || (D == 32 && KSC == 16))) ||
                !fused_width_ok(16 * KSC, sizeof(T))) {
    return hipErrorInvalidValue;
  } else {
    if (EncShape<D>::HPG > 1 && p.QB % NQW != 0) return hipErrorInvalidValue;  // one head per wave
    const int HG = p.H / EncShape<D>::HPG;
    const int64_t nck = (int64_t)p.B * p.nchunks;
    const unsigned grid = (unsigned)(((nck + 7) / 8) * 8 * HG * p.qgroups);
    const size_t lds = enc_fused_lds_bytes(16 * KSC, D, W, sizeof(T));
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_encode_fused<T, D, KSC, NQW, W>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    k_encode_fused<T, D, KSC, NQW, W><<<grid, 64 * W, lds, s>>>(p);
    return hipGetLastError();
  }
}

template <typename T, int D, int KSC, int W>
static hipError_t enc_nqw(const EncFusedParams& p, hipStream_t s) {
  switch (p.nqw) {
    case 1: return enc_one<T, D, KSC, 1, W>(p, s);
    case 2: return enc_one<T, D, KSC, 2, W>(p, s);
    case 4: return enc_one<T, D, KSC, 4, W>(p, s);
  }
  return hipErrorInvalidValue;
}

template <typename T, int D, int W>
static hipError_t enc_ksc(const EncFusedParams& p, hipStream_t s) {
  switch (p.C) {
    case 64: return enc_nqw<T, D, 4, W>(p, s);
    case 128: return enc_nqw<T, D, 8, W>(p, s);
    case 256: return enc_nqw<T, D, 16, W>(p, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_encode_fused(const EncFusedParams& p, int D, int waves, hipStream_t s) {
  if (waves == 8) {
    if (D == 16) return enc_ksc<T, 16, 8>(p, s);
    if (D == 32) return enc_ksc<T, 32, 8>(p, s);
    return hipErrorInvalidValue;
  }
  switch (D) {
    case 16: return enc_ksc<T, 16, 4>(p, s);
    case 32: return enc_ksc<T, 32, 4>(p, s);
    case 64: return enc_ksc<T, 64, 4>(p, s);
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

template <typename T, int D, int KSC>
static hipError_t dec_launch(const DecFusedParams& p, hipStream_t s) {
  if constexpr (!dec_fused_ok(sizeof(T), D, KSC) || !fused_width_ok(16 * KSC, sizeof(T))) {
    return hipErrorInvalidValue;
  } else {
    constexpr int NW = dec_waves(16 * KSC);
    const unsigned grid = (unsigned)((int64_t)p.B * ((p.N + 32 * NW - 1) / (32 * NW)));
    if constexpr (sizeof(T) == 2 && (D == 16 || D == 32) && KSC <= 8) {
      if (p.kind == kDecodePersist) {  // one persistent workgroup per CU, static LDS
        if (persist_lds_bytes(16 * KSC, D, p.Mp, sizeof(T)) > kPersistLdsBytes ||
            p.stage_bytes != (int)persist_stage_bytes(D, p.Mp, sizeof(T)))
          return hipErrorInvalidValue;
        int dev = 0, ncu = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        const unsigned pgrid = (unsigned)std::min<int64_t>((int64_t)grid, std::max(ncu, 1));
        k_decode_persist<T, D, KSC><<<pgrid, 64 * NW, 0, s>>>(p);
        return hipGetLastError();
      }
    }
    if (p.kind == kDecodePersist) return hipErrorInvalidValue;
    if constexpr (16 * KSC <= 128) {  // per-group stages (k_decode2)
      if constexpr (sizeof(T) == 2 && (D == 16 || (D == 32 && KSC <= 4))) {
        const int rt = p.Mp / 32;
        if (p.kind == kDecodeGroupsResident && rt <= 4) {
          const size_t lds = dec2_lds_bytes(16 * KSC, D, p.Mp, sizeof(T), true);
          const void* fn = rt == 1   ? reinterpret_cast<const void*>(&k_decode3<T, D, KSC, 1>)
                           : rt == 2 ? reinterpret_cast<const void*>(&k_decode3<T, D, KSC, 2>)
                           : rt == 3 ? reinterpret_cast<const void*>(&k_decode3<T, D, KSC, 3>)
                                     : reinterpret_cast<const void*>(&k_decode3<T, D, KSC, 4>);
          hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
          if (e != hipSuccess) return e;
          switch (rt) {
            case 1: k_decode3<T, D, KSC, 1><<<grid, 64 * NW, lds, s>>>(p); break;
            case 2: k_decode3<T, D, KSC, 2><<<grid, 64 * NW, lds, s>>>(p); break;
            case 3: k_decode3<T, D, KSC, 3><<<grid, 64 * NW, lds, s>>>(p); break;
            default: k_decode3<T, D, KSC, 4><<<grid, 64 * NW, lds, s>>>(p); break;
          }
          return hipGetLastError();
        }
      }
      if (p.kind != kDecodeStaged) {
        const bool res = p.kind == kDecodeGroupsResident;
        const size_t lds = dec2_lds_bytes(16 * KSC, D, p.Mp, sizeof(T), res);
        const void* fn = res ? reinterpret_cast<const void*>(&k_decode2<T, D, KSC, true>)
                             : reinterpret_cast<const void*>(&k_decode2<T, D, KSC, false>);
        hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        if (res) k_decode2<T, D, KSC, true><<<grid, 64 * NW, lds, s>>>(p);
        else k_decode2<T, D, KSC, false><<<grid, 64 * NW, lds, s>>>(p);
        return hipGetLastError();
      }
    }
    if (p.kind != kDecodeStaged) return hipErrorInvalidValue;
    {
      const size_t lds = (2 * (size_t)p.stage_elems + 16) * sizeof(T);  // + the constant rows
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_decode_fused<T, D, KSC>),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
      k_decode_fused<T, D, KSC><<<grid, 64 * NW, lds, s>>>(p);
      return hipGetLastError();
    }
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

template hipError_t launch_encode_fused<float>(const EncFusedParams&, int, int, hipStream_t);
template hipError_t launch_encode_fused<__bf16>(const EncFusedParams&, int, int, hipStream_t);
template hipError_t launch_combine_par<float>(const CombineParams&, hipStream_t);
template hipError_t launch_combine_par<__bf16>(const CombineParams&, hipStream_t);
template hipError_t launch_decode_fused<float>(const DecFusedParams&, int, hipStream_t);
template hipError_t launch_decode_fused<__bf16>(const DecFusedParams&, int, hipStream_t);

}  // namespace flarepp
