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
  // decode output: y[b*y_sb + n*y_row + h*D + d]
  void* y; int64_t y_sb, y_row;
};

struct CombineParams {
  const float* part_ml; const float* part_acc;
  int64_t BH;
  int R, M, Mp, D;
  float qscale;
  float* out32;  // [BH][M][D] or null
  float* lse;    // [BH][M] or null (natural log)
  void* q_op;    // [BH][Mp][D] scaled, or null
  void* z_op;    // [BH][D][Mp], or null
};

// ---- fused path -------------------------------------------------------------
enum FragMode { kFragPlain = 0, kFragKeyPerm = 1, kFragMerge = 2 };

struct PrepFusedParams {
  int C;
  const void* w[5];  // W_K, W_V, W~_K, W~_V, W_O  [C][C]
  void* wf[5];       // fragments [C/32][C/16][64][8]
  int mode[5];       // FragMode per weight
  const void* seeds;  // [H][M][D]
  int H, M, Mp, D;
  float qscale;
  void* seeds_op;     // [H][Mp][D] scaled
};

struct EncFusedParams {
  const void* x;                     // [B][N][C]
  const void* wkf;                   // key fragments (key-permuted)
  const void* wvf;                   // value fragments (plain)
  const void* q_op; int64_t q_sb;    // [.][H][Mp][D] scaled queries, batch stride
  int B, N, C, H, Mp, QB;
  int qgroups, chunk, nchunks;
  float fast_lim;
  float* part_ml; float* part_acc;   // [B][H][nchunks][Mp] x {2 | D}
};

struct DecFusedParams {
  const void* x;      // [B][N][C]
  const void* wkf;    // key fragments (key-permuted)
  const void* wof;    // merge fragments of W_O
  const void* q_op;   // [B][H][Mp][D] scaled synthesised queries
  const void* z_op;   // [B][H][D][Mp] latents
  int B, N, C, H, M, Mp;
  float fast_lim;
  void* y;            // [B][N][C] decoded tokens, or null
  void* o;            // [B][N][C]
  int stage_elems;    // elements per LDS stage buffer
};

// Largest number of 32-query blocks one wave of the fused encode holds
// without spilling registers (a power of two; 0: the fused encode is not
// used for this storage size, head width and C = 16 * ksc).
constexpr int enc_nqw_cap(int elem_bytes, int D, int ksc) {
  if (elem_bytes == 2) {
    if (D == 16) return ksc <= 8 ? 8 : 4;
    if (D == 32) return 4;
    return ksc <= 8 ? 2 : 0;
  }
  if (D == 16) return ksc <= 8 ? 4 : 0;
  if (D == 32) return ksc <= 4 ? 4 : (ksc <= 8 ? 2 : 0);
  return ksc <= 4 ? 1 : 0;
}
// The fused decode is used unless it would spill (fp32 with D = 64, C >= 128).
constexpr bool dec_fused_ok(int elem_bytes, int D, int ksc) { return !(elem_bytes == 4 && D == 64 && ksc >= 8); }
// The fused kernels are instantiated for these widths.
constexpr bool fused_width_ok(int C) { return C == 64 || C == 128 || C == 256; }
constexpr size_t enc_fused_lds(int C, int D, int elem_bytes) {
  return 2ull * (D == 64 ? 2 : 1) * (C / 16) * 512 * elem_bytes;
}
int decode_stage_elems(int C, int D, int Mp);
bool decode_fused_fits(int C, int D, int Mp, int elem_bytes);

template <typename T> hipError_t launch_prep_fused(const PrepFusedParams&, hipStream_t);
template <typename T> hipError_t launch_encode_fused(const EncFusedParams&, int D, int nqw, hipStream_t);
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

template <typename T> hipError_t launch_weight_frags(const WeightFragParams&, hipStream_t);
template <typename Ts, typename T> hipError_t launch_route_prep(const RoutePrepParams&, hipStream_t);
template <typename T> hipError_t launch_dmajor(const DmajorParams&, hipStream_t);
template <typename T> hipError_t launch_project(const ProjParams&, hipStream_t);
template <typename T> hipError_t launch_route(const RouteParams&, int D, bool decode, hipStream_t);

}  // namespace flarepp
