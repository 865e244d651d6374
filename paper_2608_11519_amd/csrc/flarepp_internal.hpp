// Kernel parameter blocks and launchers shared by the C ABI and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace flarepp {

enum ProjLayout { kHeadsTokenMajor = 0, kHeadsDMajor = 1, kPlain = 2 };

struct WeightFragParams {
  int C, nw;
  const void* w[5];
  void* out[5];
};

struct RoutePrepParams {
  const void* src;       // [B?][H][M][D]
  int64_t src_bstride;   // elements between batch entries (0: shared)
  int B, H, M, Mp, D;
  float qscale;
  void* q_op;            // [B][H][Mp][D] (scaled) or null
  void* z_op;            // [B][H][D][Mp] or null
};

struct DmajorParams {
  const void* src;  // [BH][N][D]
  void* dst;        // [BH][D][Np]
  int64_t BH;
  int N, Np, D;
};

struct ProjParams {
  const void* x;  // [B][N][C]
  int B, N, Np, C, H, D, nw;
  const void* wf[5];
  void* out[5];
  int layout[5];
  const void* res;  // kPlain outputs: [B][N][C] added to the product, or null
};

// Layer normalisation over the channels of every token: y = (x - mean) /
// sqrt(var + eps) * gamma + beta (biased variance), one wave per token.
struct LayerNormParams {
  const void* x; const void* gamma; const void* beta; void* y;
  int64_t T; int C;
  float eps;
  float* mean; float* rstd;  // optional [T]: each token's mean and 1 / sqrt(var + eps)
};
// Layer-norm backward of the block O = X + mixer(LN(X)): dx = dO + the
// layer norm's input gradient for the normalised-input gradient dxn (fp32);
// per token chunk, the partial sums of dgamma = sum dxn * xhat and dbeta =
// sum dxn over the chunk's tokens.
struct LayerNormBwdParams {
  const void* x; const void* gamma; const float* mean; const float* rstd;
  const float* dxn; const void* dO; float* dx;
  float* part;  // [2][nchunks][C]: dgamma partials, then dbeta partials
  int64_t T; int C; int nchunks; int64_t chunk;
};

struct RouteParams {
  // key side: rows [.. ka_rows][D] (A operand of the scores) and d-major
  // [D][va_ld] (A operand of the values), per (b, h) at b*sb + h*sh
  const void* ka; int64_t ka_sb, ka_sh; int ka_rows;
  const void* va; int64_t va_sb, va_sh; int va_ld;
  // query side: rows [.. qs_rows][D] (B operand of the scores)
  const void* qs; int64_t qs_sb, qs_sh; int qs_rows;
  int B, H;
  int key_len, key_chunk, nchunks;
  int nqb, qgroups;
  // squared bound on |score| (log2 units) below which a tile skips the running
  // maximum; negative disables that path
  float fast_lim;
  // encode output: partials [B][H][nchunks][Mp] x {(m, l), acc[D]}
  float* part_ml; float* part_acc; int Mp;
  // decode output: y[b*y_sb + n*y_row + h*D + d], and optionally each
  // token's log-normaliser over the routes in log2 units, lse2[b*H + h][n]
  void* y; int64_t y_sb, y_row;
  float* lse2;
};

struct PrepFusedParams {
  int C, nw;         // nw weights converted
  const void* w[5];  // [C][C] each
  void* wf[5];       // fragments [C/32][C/16][64][8]
  int mode[5];       // FragMode per weight
  const void* seeds;  // [H][M][D]
  int H, M, Mp, D;
  float qscale;
  int seed_copies;    // copies of the seed operand written back to back
  void* seeds_op;     // [seed_copies][H] x q fragment order, scaled
  float* qnorm2;      // [seed_copies][H][Mp / 4] max |scaled q|^2 per 4 routes, or null
};

struct CombineParams {
  const float* part_ml; const float* part_acc;
  int64_t BH;
  int R, M, Mp, D;
  float qscale;
  float* out32;  // [BH][M][D] or null
  float* lse;    // [BH][M] or null (natural log)
  // Route operands for the next call, in one of two layouts:
  //  frag == 0: q_op [BH][Mp][D] (scaled), z_op [BH][D][Mp]       (k_route)
  //  frag == 1: fragment order, see q_frag_index / z_frag_index   (fused)
  int frag;
  void* q_op;
  void* z_op;
  float* qnorm2;  // frag == 1 with q_op: [BH][Mp / 4] max of |scaled q|^2 over
                  // each group of 4 routes (one entry per wave), or null
  // the frag == 0 layouts as well, whatever frag is (the backward's unfused
  // decode after fused encodes): q_rows [BH][Mp][D] scaled, z_rows [BH][D][Mp]
  void* q_rows;
  void* z_rows;
  // fragment conversion for the later kernels (prep_n items), spread over the
  // threads: each issues its item's loads first and stores it at the end
  PrepFusedParams prep;
  int64_t prep_n;
};

// Fragment order of the route operands of the fused kernels (per (b, h)):
//  q: [Mp/32][D/16][64 lanes][8]; lane (c, g) element j = q[32 qb + c][16 js + 8 g + j]
//     (the B operand of the encode scores and the A operand of the decode scores)
//  z: [Mp/32][2 halves][RB][2 g][ZC][8] with ZC = min(D, 32) value channels c:
//     element j = z[32 rt + 16 hf + 8 (j / 4) + 4 g + j % 4][32 rb + c]
//     (the A operand of the decode value product for lanes (c, g), c < ZC; for
//     D = 16 the kernel supplies rows 16 (ones: the softmax denominators) to 31)
__host__ __device__ constexpr int64_t z_frag_elems_per_head(int Mp, int D) { return (int64_t)Mp * D; }
__host__ __device__ constexpr int64_t z_frag_index(int rt, int hf, int rb, int g, int c, int j, int D) {
  return (((((int64_t)rt * 2 + hf) * ((D + 31) / 32) + rb) * 2 + g) * (D < 32 ? D : 32) + c) * 8 + j;
}

// ---- fused path -------------------------------------------------------------
// kFragMergeHg: the kFragMerge fragments stored head-group major,
// [C/32 / (D == 64 ? 2 : 1) groups][C/32 output blocks][k steps of the group][64][8]
enum FragMode { kFragPlain = 0, kFragKeyPerm = 1, kFragMerge = 2, kFragMergeHg = 3 };


struct EncFusedParams {
  const void* x;                     // [B][N][C]
  const void* wkf;                   // key fragments (key-permuted)
  const void* wvf;                   // value fragments (plain)
  const void* q_op; int64_t q_sb;    // [.][H] x q fragment order, scaled; batch stride
  int B, N, C, H, Mp, QB;
  int nqw, qgroups, chunk, nchunks;  // query blocks per wave, query groups, tokens
                                     // per chunk (multiple of 32 * waves), chunks
  float fast_lim;
  float* part_ml; float* part_acc;   // [B][H][nchunks][Mp] x {2 | D}
  // The first routing call of a forward reads the row-major weights and the
  // learned seeds itself (wk_raw, wv_raw [C][C], seeds_raw [H][M][D]); when
  // null the fragments wkf / wvf and q_op are read.
  const void* wk_raw; const void* wv_raw;
  const void* seeds_raw;
  int M;
  float qscale;
};

struct DecFusedParams {
  const void* x;      // [B][N][C]
  const void* wkf;    // key fragments (key-permuted)
  const void* wof;    // merge fragments of W_O
  const void* q_op;   // [B][H] x q fragment order: scaled synthesised queries
  const void* z_op;   // [B][H] x z fragment order: latents
  const float* qnorm2;  // [B][H][Mp / 4] max |scaled q|^2 per group of 4 routes
  int B, N, C, H, M, Mp;
  float fast_lim;
  void* y;            // [B][N][C] decoded tokens, or null
  float* lse2;        // [B][H][N] log2 softmax normaliser of each token's scaled scores, or null
  void* o;            // [B][N][C]
  const void* res;    // [B][N][C] added to O (the block's residual), or null
  int stage_elems;    // elements per LDS stage buffer (k_decode_fused)
  int stage_bytes;    // bytes per head-group stage (k_decode2)
  int kind;           // DecodeKind
};

// Fused path coverage.  bf16: C in {64, 128, 256}; fp32 (a correctness path):
// C = 64.  Query blocks per wave of the fused encode: a power of two up to
// enc_nqw_cap (bf16 at D = 16: four, so that one eight-wave workgroup holds
// all 32 query slots of a head group at M = 512 and the K, V of a token chunk
// are projected once instead of once per query group); waves per encode
// workgroup: enc_waves (eight, two per SIMD, where the registers allow it
// with at least eight query slots).
constexpr bool fused_width_ok(int C, int elem_bytes) {
  return elem_bytes == 2 ? (C == 64 || C == 128 || C == 256) : C == 64;
}
constexpr int enc_nqw_cap(int D, int waves, int elem_bytes) {
  return D == 16 ? (waves == 8 && elem_bytes == 4 ? 2 : 4) : (D == 32 ? 2 : 1);
}
constexpr int enc_waves(int D, int C, int slots) {
  return ((D == 16 && C <= 128) || (D == 32 && C == 256)) && slots >= 8 ? 8 : 4;
}
constexpr bool dec_fused_ok(int elem_bytes, int D, int ksc) { return !(elem_bytes == 4 && D == 64 && ksc >= 8); }
size_t enc_fused_lds_bytes(int C, int D, int waves, int elem_bytes);
int decode_stage_elems(int C, int D, int Mp);
bool decode_fused_fits(int C, int D, int Mp, int elem_bytes);
// Decode kernels: k_decode_fused (per-group stages of keys and routes, W_O
// staged by output block at the end), k_decode2 with per-group stages that
// also carry the group's W_O rows (two alternating buffers, or all resident).
// k_decode_persist: persistent workgroups with W_K and W_O resident in LDS and
// the route operands of one head at a time in two alternating stages.
enum DecodeKind { kDecodeStaged = 0, kDecodeGroupsStaged = 1, kDecodeGroupsResident = 2, kDecodePersist = 3 };
int decode_kind(int C, int D, int Mp, int elem_bytes);
bool decode_kind_fits(int kind, int C, int D, int Mp, int elem_bytes);
size_t persist_stage_bytes(int D, int Mp, int elem_bytes);
size_t persist_lds_bytes(int C, int D, int Mp, int elem_bytes);
constexpr size_t kPersistLdsBytes = 160 * 1024;  // static LDS of k_decode_persist
size_t dec2_stage_bytes(int C, int D, int Mp, int elem_bytes);
size_t dec2_lds_bytes(int C, int D, int Mp, int elem_bytes, bool res);

// Items of work (fragment lanes, seed operand lanes, norm bounds) in a prep.
int64_t prep_fused_items(const PrepFusedParams& p);
template <typename T> hipError_t launch_encode_fused(const EncFusedParams&, int D, int waves, hipStream_t);
template <typename T> hipError_t launch_combine_par(const CombineParams&, hipStream_t);
template <typename T> hipError_t launch_decode_fused(const DecFusedParams&, int D, hipStream_t);

// Exponent range (log2 units) inside which the softmax runs without a running
// maximum: with |t| <= 64 every 2^t, every row sum over 2^20+ keys and every
// weighted sum of values stays a normal fp32 number.
constexpr float kFastRangeSq = 64.0f * 64.0f;

// Query blocks (of 32) held per wave by k_route.
constexpr int route_nq(int D, bool decode) {
  return decode ? (D <= 32 ? 2 : 1) : (D == 16 ? 4 : (D == 32 ? 2 : 1));
}

// ---- backward (App. A.5) ---------------------------------------------------
// C[M][N] = sum over segments of sum_k A(m, k) B(k, n) (A, B in T), with
// A(m, k) = a[m * a_m + k * a_k] and B(k, n) = b[k * b_k + n * b_n] (elements).
// Either nseg segments accumulate into one product (nprob = 1), or nprob
// independent products of one segment each share the shapes and strides.
// Split-K: product p, split z covers k in [z * kchunk, (z + 1) * kchunk) and
// writes c + (p * splits + z) * split_stride (fp32), or, with c_t and a
// single split, the compute type T.
struct GemmParams {
  int M, N, K, nseg, nprob, splits;
  const void* a[16];  // operands of segment j of problem i at [i * nseg + j];
  const void* b[16];  // a null b after the first segment ends the problem's list
  int64_t a_m, a_k, b_k, b_n;
  int kchunk;
  void* c;
  int c_t;
  int64_t ldc, split_stride;
};

// SDPA backward over one (batch, head) pair and one chunk of the long axis
// (keys of an encode, tokens of the decode).  The tile orientation is
// rows = short axis (the M routes), columns = long axis, so that
//   S = A_sh B_lo^T, dP = G_sh G_lo^T, dS = P (dP - c),
//   long side:  dB_lo^T = s A_sh^T dS (both),  dG_lo^T = G_sh^T P (encode),
//   short side: dA_sh = s dS B_lo (both),      dG_sh = P G_lo (decode).
// Encode: A_sh = queries, G_sh = dOut, B_lo = keys, G_lo = values, L and c
// per route.  Decode: A_sh = routes (its keys), G_sh = latents (its values),
// B_lo = token keys (its queries), G_lo = dY, L per token from the forward
// and c per token computed in the kernel.
struct AttnBwdParams {
  int B, H, Nl, M, Mp, R, tpw;   // long length, routes, chunks per (b, h), long tiles per wave
  int sb0, nsb;                  // the window of route blocks [sb0, sb0 + nsb) of this launch
  float s, sl2;                  // 1/sqrt(D), and times log2(e) (the route rows ash come scaled by sl2)
  // short side, per (b, h) at b * sb + h * sh (elements)
  const void* ash; int64_t ash_sb, ash_sh;    // rows [Mp][D]
  const void* asht; int64_t asht_sb, asht_sh; // A fragments of A_sh^T
  const void* gsh; int64_t gsh_sb, gsh_sh;    // rows [Mp][D]
  const void* gsht; int64_t gsht_sb, gsht_sh; // A fragments of G_sh^T (encode)
  const float* lrow;  // encode: [B * H][Mp], log-normaliser in log2 units
  const float* crow;  // encode: [B * H][Mp]
  // long side: element (b, h, n, d) at b * sb + h * sh + n * sn + d * sd
  const void* blo; int64_t blo_sb, blo_sh, blo_sn, blo_sd;  // type T
  const void* glo; int64_t glo_sb, glo_sh, glo_sn, glo_sd;  // type T
  const void* ylo; int64_t ylo_sb, ylo_sh, ylo_sn;          // decode: forward output rows (T)
  const float* lcol;  // decode: [B * H][Nl], each position's log-normaliser in log2 units
  // outputs: long side [B][Nl][H * D] in T (added to what is there when
  // acc_b / acc_g); short side partials [B][H][R][Mp][D] fp32 (this window's
  // rows).  With dout_b_lo / dout_g_lo (bf16 only) a long-side value v is
  // kept as hi = bf16(v) in dout and lo = bf16(v - hi) there, and read back
  // as hi + lo
  void* dout_b; void* dout_b_lo; int acc_b;
  void* dout_g; void* dout_g_lo; int acc_g;
  float* part_a; float* part_g;
};
// LDS of a launch over a window of nsb route blocks (Mp routes in all)
int attn_bwd_waves(int D, int nsb, int Mp, bool dec, int elem_bytes);
size_t attn_bwd_lds_bytes(int D, int nsb, int Mp, bool dec, int waves, int elem_bytes);

// Fixed-order sums of backward partials: out[o][m][d] = base[o][m][d] +
// sum_{p < P} (sum_{r < R0} part0[p][o][r][m][d] + sum_{r < R1} part1[p][o][r][m][d]),
// partials laid out [P][O][R][Mp][D] fp32 (part1 and base optional).
struct BwdReduceParams {
  const float* part0; int R0;
  const float* part1; int R1;
  const float* base; float* out;
  int P, O, M, Mp, D;
};
// Short-side operands of a backward call from rows src[O][M][D] (fp32 or T),
// each output optional: T rows [O][Mp][D] (zero padded); the A fragments of
// src^T [O][Mp / 32][2][DB][64][8] (lane (c, g), element j holds
// src[32 sb + 16 kk + acc_row16(g, j)][32 db + c]); c[O][Mp] = sum_d
// src[m][d] dot[m][d]; l2[O][Mp] = lse[O][M] * log2(e) (zero padded).  Up to
// three jobs run in one launch.
struct BwdPrepJob {
  const void* src; int src_is_f32;
  const float* dot;
  const float* lse;
  int O;
  void* rows; void* tfrag; float* c; float* l2;
  float rows_scale;  // rows are stored times this (0 is taken as 1)
};
struct BwdPrepParams {
  int M, Mp, D, njobs;
  BwdPrepJob job[3];
};
template <typename T> hipError_t launch_gemm(const GemmParams&, hipStream_t);
template <typename T> hipError_t launch_attn_bwd(const AttnBwdParams&, int D, bool dec, hipStream_t);
// out[p][i] = sum_z part[(p * splits + z) * n + i], p < nprob (at most 5)
hipError_t launch_sum_splits(const float* part, float* const* out, int64_t n, int splits, int nprob, hipStream_t);
hipError_t launch_bwd_reduce(const BwdReduceParams&, hipStream_t);
template <typename T> hipError_t launch_bwd_prep(const BwdPrepParams&, hipStream_t);
int64_t bwd_prep_items(const BwdPrepParams&, int job);

template <typename T> hipError_t launch_layernorm(const LayerNormParams&, hipStream_t);
template <typename T> hipError_t launch_layernorm_bwd(const LayerNormBwdParams&, hipStream_t);
template <typename T> hipError_t launch_weight_frags(const WeightFragParams&, hipStream_t);
template <typename Ts, typename T> hipError_t launch_route_prep(const RoutePrepParams&, hipStream_t);
template <typename T> hipError_t launch_dmajor(const DmajorParams&, hipStream_t);
template <typename T> hipError_t launch_project(const ProjParams&, hipStream_t);
template <typename T> hipError_t launch_route(const RouteParams&, int D, bool decode, hipStream_t);

}  // namespace flarepp
