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
template <typename T> hipError_t launch_combine(const CombineParams&, hipStream_t);
template <typename T> hipError_t launch_route(const RouteParams&, int D, bool decode, hipStream_t);

}  // namespace flarepp
