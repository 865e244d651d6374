// C ABI of libflarepp.so: argument validation, workspace layout and launch
// sequencing for the FLARE++ mixer forward.  Declarations and the contract
// of every entry point are in include/flarepp.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <mutex>
#include <string>
#include <type_traits>
#include <algorithm>

#include "../../include/flarepp.h"
#include "flarepp_internal.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int ok() {
  g_last_error.clear();
  return FLAREPP_OK;
}

constexpr int64_t kMaxTokens = int64_t(1) << 30;  // per batch entry
constexpr int64_t kMaxRoutes = 1 << 16;
constexpr int64_t kMaxWidth = 4096;
constexpr int64_t kTargetUnits = 2048;  // waves per encode launch (8 per CU)
constexpr int kMinChunk = 128;          // tokens per encode unit
constexpr int64_t kFusedEncWaves = 2048;  // waves per fused encode launch (8 per CU)

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int dtype_bytes(int dtype) { return dtype == FLAREPP_F32 ? 4 : 2; }

int check_dtype(int dtype) {
  if (dtype != FLAREPP_F32 && dtype != FLAREPP_BF16)
    return fail(FLAREPP_ERR_UNSUPPORTED, "unknown dtype %d (expected FLAREPP_F32=0 or FLAREPP_BF16=1)", dtype);
  return FLAREPP_OK;
}

int check_head_width(int64_t D) {
  if (D != 16 && D != 32 && D != 64)
    return fail(FLAREPP_ERR_UNSUPPORTED, "head width D=%lld is not supported (16, 32 or 64)", (long long)D);
  return FLAREPP_OK;
}

int check_ptr(const void* p, const char* name, bool may_be_null = false) {
  if (!p) {
    if (may_be_null) return FLAREPP_OK;
    return fail(FLAREPP_ERR_INVALID_ARG, "%s is NULL", name);
  }
  if (reinterpret_cast<uintptr_t>(p) & 15)
    return fail(FLAREPP_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return FLAREPP_OK;
}

int check_positive(int64_t v, const char* name) {
  if (v < 1) return fail(FLAREPP_ERR_INVALID_ARG, "%s=%lld must be >= 1", name, (long long)v);
  return FLAREPP_OK;
}

#define TRY(x) do { int _rc = (x); if (_rc != FLAREPP_OK) return _rc; } while (0)
#define HIPTRY(x) do { hipError_t _e = (x); if (_e != hipSuccess) \
    return fail(FLAREPP_ERR_HIP, "%s: %s", #x, hipGetErrorString(_e)); } while (0)

int check_mixer_shape(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  TRY(check_dtype(dtype));
  TRY(check_positive(B, "B"));
  TRY(check_positive(N, "N"));
  TRY(check_positive(C, "C"));
  TRY(check_positive(H, "H"));
  TRY(check_positive(M, "M"));
  if (C % H) return fail(FLAREPP_ERR_INVALID_ARG, "C=%lld is not divisible by H=%lld", (long long)C, (long long)H);
  TRY(check_head_width(C / H));
  if (C % 32) return fail(FLAREPP_ERR_UNSUPPORTED, "C=%lld must be a multiple of 32", (long long)C);
  if (N > kMaxTokens) return fail(FLAREPP_ERR_UNSUPPORTED, "N=%lld exceeds %lld", (long long)N, (long long)kMaxTokens);
  if (M > kMaxRoutes) return fail(FLAREPP_ERR_UNSUPPORTED, "M=%lld exceeds %lld", (long long)M, (long long)kMaxRoutes);
  if (C > kMaxWidth) return fail(FLAREPP_ERR_UNSUPPORTED, "C=%lld exceeds %lld", (long long)C, (long long)kMaxWidth);
  if (B * H > (int64_t(1) << 24)) return fail(FLAREPP_ERR_UNSUPPORTED, "B*H too large");
  if (B * round_up(N, 32) * C > (int64_t(1) << 40)) return fail(FLAREPP_ERR_UNSUPPORTED, "B*N*C too large");
  return FLAREPP_OK;
}

// ---- encode work split ----------------------------------------------------
struct EncPlan {
  int nq, nqb, qgroups, nchunks, chunk;
};

EncPlan encode_plan(int64_t B, int64_t H, int64_t N, int64_t Mp, int64_t D) {
  EncPlan e;
  e.nq = flarepp::route_nq((int)D, false);
  e.nqb = (int)(Mp / 32);
  e.qgroups = (int)cdiv(e.nqb, e.nq);
  const int64_t per = B * H * e.qgroups;
  int64_t R;
  const char* force = std::getenv("FLAREPP_FORCE_CHUNKS");
  const int64_t forced = force ? std::atoll(force) : 0;
  if (forced > 0) {
    R = forced > 65536 ? 65536 : forced;
    e.chunk = (int)round_up(cdiv(N, R), 32);
  } else {
    R = cdiv(kTargetUnits, per);
    R = std::max<int64_t>(1, std::min<int64_t>(R, cdiv(N, kMinChunk)));
    e.chunk = (int)round_up(cdiv(N, R), 32);
    R = cdiv(N, e.chunk);
  }
  e.nchunks = (int)R;
  return e;
}

// Decode kernel for a shape; FLAREPP_DECODE_KIND (0, 1, 2) may force a
// smaller-footprint kernel than the one chosen (for testing every kernel).
int decode_kind_for(int C, int D, int Mp, int elem_bytes) {
  int k = flarepp::decode_kind(C, D, Mp, elem_bytes);
  const char* f = std::getenv("FLAREPP_DECODE_KIND");
  if (f) {
    const int want = std::atoi(f);
    if (want >= 0 && want <= flarepp::kDecodePersist && flarepp::decode_kind_fits(want, C, D, Mp, elem_bytes)) k = want;
  }
  return k;
}

// Squared score bound of the shift-free softmax path (2% below kFastRange^2
// for the rounding of the norms); FLAREPP_NO_FAST_PATH=1 disables the path.
float fast_limit() {
  const char* off = std::getenv("FLAREPP_NO_FAST_PATH");
  if (off && std::atoi(off) != 0) return -1.f;
  return flarepp::kFastRangeSq * 0.98f;
}

flarepp::RouteParams encode_params(const EncPlan& e, int64_t B, int64_t H, int64_t N, int64_t Mp,
                                   int64_t D) {
  flarepp::RouteParams p{};
  p.B = (int)B;
  p.H = (int)H;
  p.key_len = (int)N;
  p.key_chunk = e.chunk;
  p.nchunks = e.nchunks;
  p.nqb = e.nqb;
  p.qgroups = e.qgroups;
  p.Mp = (int)Mp;
  p.fast_lim = fast_limit();
  (void)D;
  return p;
}

flarepp::RouteParams decode_params(int64_t B, int64_t H, int64_t N, int64_t M, int64_t D) {
  flarepp::RouteParams p{};
  const int nq = flarepp::route_nq((int)D, true);
  p.B = (int)B;
  p.H = (int)H;
  p.key_len = (int)M;
  p.key_chunk = (int)round_up(M, 32);
  p.nchunks = 1;
  p.nqb = (int)cdiv(N, 32);
  p.qgroups = (int)cdiv(p.nqb, nq);
  p.fast_lim = fast_limit();
  return p;
}

// ---- workspace carving ----------------------------------------------------
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  }
};

// ---- mixer plan ------------------------------------------------------------
struct MixerPlan {
  bool fused;
  EncPlan enc;   // unfused split (k_route)
  // fused split (k_encode_fused)
  int waves, nqw, qgroups, nchunks, chunk;
};

int64_t next_pow2(int64_t x) {
  int64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

MixerPlan mixer_plan(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  MixerPlan pl{};
  const int64_t D = C / H, Mp = round_up(M, 32), bs = dtype_bytes(dtype);
  const int ksc = (int)(C / 16);
  const int64_t hpg = D == 16 ? 2 : 1, slots = hpg * (Mp / 32);
  pl.waves = flarepp::enc_waves((int)D, (int)C, (int)slots);
  const char* off = std::getenv("FLAREPP_UNFUSED");
  pl.fused = flarepp::fused_width_ok((int)C, (int)bs) && flarepp::dec_fused_ok((int)bs, (int)D, ksc) &&
             flarepp::decode_fused_fits((int)C, (int)D, (int)Mp, (int)bs) &&
             flarepp::enc_fused_lds_bytes((int)C, (int)D, pl.waves, (int)bs) <= 160 * 1024 &&
             !(off && std::atoi(off) != 0);
  pl.enc = encode_plan(B, H, N, Mp, D);
  if (pl.fused) {
    pl.nqw = (int)std::min<int64_t>(flarepp::enc_nqw_cap((int)D, pl.waves, (int)bs), next_pow2(cdiv(slots, pl.waves)));
    // every wave's query slots must belong to one head of the group
    while (hpg > 1 && (Mp / 32) % pl.nqw != 0) pl.nqw /= 2;
    pl.qgroups = (int)cdiv(slots, (int64_t)pl.waves * pl.nqw);
    const int64_t per = B * (H / hpg) * pl.qgroups;  // workgroups per token chunk
    const int64_t step = 32 * pl.waves;                // tokens per workgroup step
    const char* force = std::getenv("FLAREPP_FORCE_CHUNKS");
    const int64_t forced = force ? std::atoll(force) : 0;
    int64_t R;
    if (forced > 0) {
      R = std::min<int64_t>(forced, 65536);
      pl.chunk = (int)round_up(cdiv(N, R), step);
    } else {
      const char* tw = std::getenv("FLAREPP_ENC_WAVES");
      const int64_t target = tw && std::atoll(tw) > 0 ? std::atoll(tw) : kFusedEncWaves;
      R = std::max<int64_t>(1, std::min<int64_t>(cdiv(target / pl.waves, per), cdiv(N, step)));
      pl.chunk = (int)round_up(cdiv(N, R), step);
      R = cdiv(N, pl.chunk);
    }
    pl.nchunks = (int)R;
  }
  return pl;
}

struct MixerWs {
  void *wf[5], *seeds_op, *K, *Kt, *Vdm, *Vtdm, *q_op, *z_op, *Y;
  float *part_ml, *part_acc;
  float* qnorm2;
  size_t bytes;
};

// flare: the fixed-query mixer (no query synthesis): no W~ fragments, no K~
// or V~, and on the fused path the seed operand is copied per batch entry
// (the decode reads route operands per batch entry).
MixerWs mixer_ws(void* base, int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                 const MixerPlan& pl, bool flare = false) {
  const int64_t D = C / H, Mp = round_up(M, 32), Np = round_up(N, 32);
  const size_t bs = dtype_bytes(dtype);
  const int64_t R = pl.fused ? pl.nchunks : pl.enc.nchunks;
  Carver cv(base);
  MixerWs w{};
  for (int i = 0; i < 5; ++i) w.wf[i] = (flare && (i == 2 || i == 3)) ? nullptr : cv.take(bs * C * C);
  // seed operand: the unfused path's (shared by the batch), or on the fused
  // fixed-query path one per batch entry (FLARE++'s first call reads the seeds)
  w.seeds_op = pl.fused && !flare ? nullptr : cv.take(bs * (flare && pl.fused ? B : 1) * H * Mp * D);
  if (!pl.fused) {
    w.K = cv.take(bs * B * H * N * D);
    w.Kt = flare ? nullptr : cv.take(bs * B * H * N * D);
    w.Vdm = cv.take(bs * B * H * D * Np);
    w.Vtdm = flare ? nullptr : cv.take(bs * B * H * D * Np);
    w.Y = cv.take(bs * B * N * C);
  }
  w.part_ml = (float*)cv.take(sizeof(float) * R * B * H * Mp * 2);
  w.part_acc = (float*)cv.take(sizeof(float) * R * B * H * Mp * D);
  w.q_op = flare ? nullptr : cv.take(bs * B * H * Mp * D);
  w.z_op = cv.take(bs * B * H * (pl.fused ? flarepp::z_frag_elems_per_head((int)Mp, (int)D) : D * Mp));
  w.qnorm2 = (float*)cv.take(sizeof(float) * B * H * (Mp / 4));
  w.bytes = cv.off;
  return w;
}

float route_qscale(int64_t D) { return (float)(1.4426950408889634 / std::sqrt((double)D)); }

// The FLARE++ mixer (Sec. 3.2, Eqs. (7)-(11)) or, with flare, the
// fixed-query FLARE mixer (Sec. 3.1, Eqs. (4)-(5)): the seeds are then the
// learned queries Q_h of both routing calls, and call 1 (stages 3 and 4) and
// the W~ projections are absent.
template <typename T>
int mixer_impl(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M, const void* X,
               const void* Wk, const void* Wv, const void* Wkt, const void* Wvt, const void* Wo,
               const void* seeds, void* O, float* Q_out, float* Z_out, void* Y_out, void* ws,
               size_t ws_bytes, hipStream_t s, hipEvent_t const* ev, int only, bool flare,
               const void* res = nullptr) {
  using namespace flarepp;
  const int64_t D = C / H, Mp = round_up(M, 32), Np = round_up(N, 32);
  const MixerPlan pl = mixer_plan(dtype, B, N, C, H, M);
  const MixerWs w = mixer_ws(ws, dtype, B, N, C, H, M, pl, flare);
  if (ws_bytes < w.bytes)
    return fail(FLAREPP_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, w.bytes);
  const float qscale = route_qscale(D);
#define STAGE(i) do { if (ev) HIPTRY(hipEventRecord(ev[i], s)); } while (0)
#define RUN(i) (only == 0 || only == (i))
  STAGE(0);
  if (pl.fused) {
    // weights as fused-path fragments and the seed operand
    // The first routing call reads the row-major weights and the seeds itself;
    // the first combine converts what the later kernels read into fragment
    // order: W_K and W_O for the decode, W_V for the second encode of
    // FLARE++, and for the fixed queries of FLARE (the decode's routes too)
    // a seed operand per batch entry with its route-norm bounds (on FLARE++
    // the combine of call 1 writes both from Q(X)).  Stages 1 and 2 launch
    // nothing.
    PrepFusedParams pp{};
    pp.C = (int)C;
    const int dkind = decode_kind_for((int)C, (int)D, (int)Mp, (int)dtype_bytes(dtype));
    const int merge_mode = dkind == kDecodeStaged ? kFragMerge : kFragMergeHg;
    auto add = [&](const void* wt, int slot, int mode) {
      pp.w[pp.nw] = wt; pp.wf[pp.nw] = w.wf[slot]; pp.mode[pp.nw] = mode; ++pp.nw;
    };
    add(Wk, 0, kFragKeyPerm);
    if (!flare) add(Wv, 1, kFragPlain);
    add(Wo, 4, merge_mode);
    pp.seeds = seeds; pp.H = (int)H; pp.M = (int)M; pp.Mp = (int)Mp; pp.D = (int)D;
    pp.qscale = qscale; pp.seeds_op = w.seeds_op;
    pp.seed_copies = flare ? (int)B : 0;
    pp.qnorm2 = flare ? w.qnorm2 : nullptr;
    STAGE(1);
    STAGE(2);  // the projections run inside the routing kernels
    EncFusedParams ep{};
    ep.x = X; ep.wk_raw = flare ? Wk : Wkt; ep.wv_raw = flare ? Wv : Wvt; ep.seeds_raw = seeds;
    ep.q_sb = 0; ep.M = (int)M; ep.qscale = qscale;
    ep.B = (int)B; ep.N = (int)N; ep.C = (int)C; ep.H = (int)H; ep.Mp = (int)Mp; ep.QB = (int)(Mp / 32);
    ep.nqw = pl.nqw; ep.qgroups = pl.qgroups; ep.chunk = pl.chunk; ep.nchunks = pl.nchunks;
    ep.fast_lim = fast_limit(); ep.part_ml = w.part_ml; ep.part_acc = w.part_acc;
    if (!flare && RUN(3)) HIPTRY(launch_encode_fused<T>(ep, (int)D, pl.waves, s));  // call 1
    STAGE(3);
    CombineParams cp{};
    cp.part_ml = w.part_ml; cp.part_acc = w.part_acc; cp.BH = B * H; cp.R = pl.nchunks;
    cp.M = (int)M; cp.Mp = (int)Mp; cp.D = (int)D; cp.qscale = qscale; cp.frag = 1;
    cp.out32 = Q_out; cp.q_op = w.q_op; cp.qnorm2 = w.qnorm2;
    cp.prep = pp; cp.prep_n = prep_fused_items(pp);
    if (!flare && RUN(4)) HIPTRY(launch_combine_par<T>(cp, s));
    STAGE(4);
    if (!flare) {  // call 2 reads the fragments the first combine wrote and Q(X)
      ep.wk_raw = ep.wv_raw = ep.seeds_raw = nullptr;
      ep.wkf = w.wf[0]; ep.wvf = w.wf[1]; ep.q_op = w.q_op; ep.q_sb = H * Mp * D;
      cp.prep_n = 0;
    }
    if (RUN(5)) HIPTRY(launch_encode_fused<T>(ep, (int)D, pl.waves, s));  // call 2 / FLARE encode
    STAGE(5);
    cp.out32 = Z_out; cp.q_op = nullptr; cp.qnorm2 = nullptr; cp.z_op = w.z_op;
    if (RUN(6)) HIPTRY(launch_combine_par<T>(cp, s));
    STAGE(6);
    DecFusedParams dp{};
    dp.x = X; dp.wkf = w.wf[0]; dp.wof = w.wf[4]; dp.q_op = flare ? w.seeds_op : w.q_op;
    dp.z_op = w.z_op; dp.qnorm2 = w.qnorm2;
    dp.B = (int)B; dp.N = (int)N; dp.C = (int)C; dp.H = (int)H; dp.M = (int)M; dp.Mp = (int)Mp;
    dp.fast_lim = fast_limit(); dp.y = Y_out; dp.o = O; dp.res = res;
    dp.stage_elems = decode_stage_elems((int)C, (int)D, (int)Mp);
    dp.stage_bytes = (int)(dkind == kDecodePersist ? persist_stage_bytes((int)D, (int)Mp, (int)dtype_bytes(dtype))
                                                   : dec2_stage_bytes((int)C, (int)D, (int)Mp, (int)dtype_bytes(dtype)));
    dp.kind = dkind;
    if (RUN(7)) HIPTRY(launch_decode_fused<T>(dp, (int)D, s));  // call 3 + merge
    STAGE(7);
    STAGE(8);
    return ok();
  }

  // 1. weights as MFMA fragments
  WeightFragParams wp{};
  wp.C = (int)C;
  const void* ws_in[5] = {Wk, Wv, Wkt, Wvt, Wo};
  for (int i = 0; i < 5; ++i) {
    if (flare && (i == 2 || i == 3)) continue;
    wp.w[wp.nw] = ws_in[i]; wp.out[wp.nw] = w.wf[i]; ++wp.nw;
  }
  if (RUN(1)) HIPTRY(launch_weight_frags<T>(wp, s));

  // 2. seeds -> scaled route operand (shared by the batch)
  RoutePrepParams sp{};
  sp.src = seeds; sp.src_bstride = 0; sp.B = 1; sp.H = (int)H; sp.M = (int)M; sp.Mp = (int)Mp;
  sp.D = (int)D; sp.qscale = qscale; sp.q_op = w.seeds_op; sp.z_op = nullptr;
  if (RUN(1)) HIPTRY((launch_route_prep<T, T>(sp, s)));
  STAGE(1);

  // 3. project: K, K~ token-major; V, V~ d-major (value operands)
  ProjParams pp{};
  pp.x = X; pp.B = (int)B; pp.N = (int)N; pp.Np = (int)Np; pp.C = (int)C; pp.H = (int)H; pp.D = (int)D;
  pp.nw = flare ? 2 : 4;
  pp.wf[0] = w.wf[0]; pp.out[0] = w.K;    pp.layout[0] = kHeadsTokenMajor;
  pp.wf[1] = w.wf[1]; pp.out[1] = w.Vdm;  pp.layout[1] = kHeadsDMajor;
  pp.wf[2] = w.wf[2]; pp.out[2] = w.Kt;   pp.layout[2] = kHeadsTokenMajor;
  pp.wf[3] = w.wf[3]; pp.out[3] = w.Vtdm; pp.layout[3] = kHeadsDMajor;
  if (RUN(2)) HIPTRY(launch_project<T>(pp, s));
  STAGE(2);

  const EncPlan e = pl.enc;
  const int64_t tokHS = N * D, tokBS = H * N * D;          // token-major strides
  const int64_t dmHS = D * Np, dmBS = H * D * Np;          // d-major token strides
  const int64_t rtHS = Mp * D, rtBS = H * Mp * D;          // route operand strides

  // 4. call 1: Q = SDPA(Q~, K~, V~), softmax over tokens
  RouteParams r1 = encode_params(e, B, H, N, Mp, D);
  r1.ka = w.Kt; r1.ka_sb = tokBS; r1.ka_sh = tokHS; r1.ka_rows = (int)N;
  r1.va = w.Vtdm; r1.va_sb = dmBS; r1.va_sh = dmHS; r1.va_ld = (int)Np;
  r1.qs = w.seeds_op; r1.qs_sb = 0; r1.qs_sh = rtHS; r1.qs_rows = (int)Mp;
  r1.part_ml = w.part_ml; r1.part_acc = w.part_acc;
  if (!flare && RUN(3)) HIPTRY(launch_route<T>(r1, (int)D, false, s));
  STAGE(3);
  CombineParams c1{};
  c1.part_ml = w.part_ml; c1.part_acc = w.part_acc; c1.BH = B * H; c1.R = e.nchunks;
  c1.M = (int)M; c1.Mp = (int)Mp; c1.D = (int)D; c1.qscale = qscale;
  c1.out32 = Q_out; c1.lse = nullptr; c1.q_op = w.q_op; c1.z_op = nullptr;
  if (!flare && RUN(4)) HIPTRY(launch_combine_par<T>(c1, s));
  STAGE(4);

  // 5. call 2: Z = SDPA(Q, K, V), softmax over tokens (FLARE: the learned
  // queries, shared by the batch)
  RouteParams r2 = r1;
  r2.ka = w.K; r2.va = w.Vdm;
  r2.qs = flare ? w.seeds_op : w.q_op; r2.qs_sb = flare ? 0 : rtBS; r2.qs_sh = rtHS; r2.qs_rows = (int)Mp;
  if (RUN(5)) HIPTRY(launch_route<T>(r2, (int)D, false, s));
  STAGE(5);
  CombineParams c2 = c1;
  c2.out32 = Z_out; c2.q_op = nullptr; c2.z_op = w.z_op;
  if (RUN(6)) HIPTRY(launch_combine_par<T>(c2, s));
  STAGE(6);

  // 6. call 3: Y = SDPA(K, Q, Z), softmax over routes, heads merged
  void* Y = Y_out ? Y_out : w.Y;
  RouteParams r3 = decode_params(B, H, N, M, D);
  r3.ka = flare ? w.seeds_op : w.q_op; r3.ka_sb = flare ? 0 : rtBS; r3.ka_sh = rtHS; r3.ka_rows = (int)Mp;
  r3.va = w.z_op; r3.va_sb = H * D * Mp; r3.va_sh = D * Mp; r3.va_ld = (int)Mp;
  r3.qs = w.K; r3.qs_sb = tokBS; r3.qs_sh = tokHS; r3.qs_rows = (int)N;
  r3.y = Y; r3.y_sb = N * C; r3.y_row = C;
  if (RUN(7)) HIPTRY(launch_route<T>(r3, (int)D, true, s));
  STAGE(7);

  // 7. merge: O = Y W_O
  ProjParams mp{};
  mp.x = Y; mp.B = (int)B; mp.N = (int)N; mp.Np = (int)Np; mp.C = (int)C; mp.H = (int)H; mp.D = (int)D;
  mp.nw = 1; mp.wf[0] = w.wf[4]; mp.out[0] = O; mp.layout[0] = kPlain; mp.res = res;
  if (RUN(8)) HIPTRY(launch_project<T>(mp, s));
  STAGE(8);
#undef RUN
#undef STAGE
  return ok();
}

int mixer_entry(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M, const void* X,
                const void* Wk, const void* Wv, const void* Wkt, const void* Wvt, const void* Wo,
                const void* seeds, void* O, float* Q_out, float* Z_out, void* Y_out, void* ws,
                size_t ws_bytes, void* stream, void* const* events, int n_events, int only = 0,
                bool flare = false) {
  TRY(check_mixer_shape(dtype, B, N, C, H, M));
  if (only < 0 || only > FLAREPP_PROFILE_EVENTS - 1)
    return fail(FLAREPP_ERR_INVALID_ARG, "stage=%d must be in [1, %d]", only, FLAREPP_PROFILE_EVENTS - 1);
  if (n_events != 0 && n_events != FLAREPP_PROFILE_EVENTS)
    return fail(FLAREPP_ERR_INVALID_ARG, "n_events=%d must be 0 or %d", n_events, FLAREPP_PROFILE_EVENTS);
  if (n_events) {
    if (!events) return fail(FLAREPP_ERR_INVALID_ARG, "events is NULL");
    for (int i = 0; i < n_events; ++i)
      if (!events[i]) return fail(FLAREPP_ERR_INVALID_ARG, "events[%d] is NULL", i);
  }
  hipEvent_t const* ev = n_events ? reinterpret_cast<hipEvent_t const*>(events) : nullptr;
  TRY(check_ptr(X, "X"));
  TRY(check_ptr(Wk, "Wk"));
  TRY(check_ptr(Wv, "Wv"));
  if (!flare) {
    TRY(check_ptr(Wkt, "Wkt"));
    TRY(check_ptr(Wvt, "Wvt"));
  }
  TRY(check_ptr(Wo, "Wo"));
  TRY(check_ptr(seeds, flare ? "queries" : "seeds"));
  TRY(check_ptr(O, "O"));
  TRY(check_ptr(Q_out, "Q_out", true));
  TRY(check_ptr(Z_out, "Z_out", true));
  TRY(check_ptr(Y_out, "Y_out", true));
  if (!ws) return fail(FLAREPP_ERR_WORKSPACE, "workspace is NULL");
  TRY(check_ptr(ws, "ws"));
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == FLAREPP_F32)
    return mixer_impl<float>(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, O, Q_out, Z_out,
                             Y_out, ws, ws_bytes, s, ev, only, flare);
  return mixer_impl<__bf16>(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, O, Q_out, Z_out,
                            Y_out, ws, ws_bytes, s, ev, only, flare);
}

// ---- route ------------------------------------------------------------------
struct RouteWs {
  void *q_op, *z_op, *Vdm;
  float *part_ml, *part_acc;
  size_t bytes;
};

RouteWs route_ws(void* base, int kind, int dtype, int64_t B, int64_t H, int64_t N, int64_t M, int64_t D,
                 bool shared_routes) {
  const int64_t Mp = round_up(M, 32), Np = round_up(N, 32);
  const size_t bs = dtype_bytes(dtype);
  const int64_t Br = shared_routes ? 1 : B;
  Carver cv(base);
  RouteWs w{};
  w.q_op = cv.take(bs * Br * H * Mp * D);
  if (kind == FLAREPP_ENCODE) {
    const EncPlan e = encode_plan(B, H, N, Mp, D);
    w.Vdm = cv.take(bs * B * H * D * Np);
    w.part_ml = (float*)cv.take(sizeof(float) * e.nchunks * B * H * Mp * 2);
    w.part_acc = (float*)cv.take(sizeof(float) * e.nchunks * B * H * Mp * D);
  } else {
    w.z_op = cv.take(bs * Br * H * D * Mp);
  }
  w.bytes = cv.off;
  return w;
}

int check_route_shape(int kind, int dtype, int64_t B, int64_t H, int64_t N, int64_t M, int64_t D) {
  if (kind != FLAREPP_ENCODE && kind != FLAREPP_DECODE)
    return fail(FLAREPP_ERR_UNSUPPORTED, "unknown route kind %d", kind);
  TRY(check_dtype(dtype));
  TRY(check_positive(B, "B"));
  TRY(check_positive(H, "H"));
  TRY(check_positive(N, "N"));
  TRY(check_positive(M, "M"));
  TRY(check_positive(D, "D"));
  TRY(check_head_width(D));
  if (N > kMaxTokens) return fail(FLAREPP_ERR_UNSUPPORTED, "N too large");
  if (M > kMaxRoutes) return fail(FLAREPP_ERR_UNSUPPORTED, "M too large");
  if (B * H > (int64_t(1) << 24)) return fail(FLAREPP_ERR_UNSUPPORTED, "B*H too large");
  return FLAREPP_OK;
}

template <typename T>
int route_impl(int kind, int dtype, int64_t B, int64_t H, int64_t N, int64_t M, int64_t D,
               const void* q, int64_t rstride, const void* k, const void* v, void* out, float* lse,
               void* ws, size_t ws_bytes, hipStream_t s) {
  using namespace flarepp;
  const bool shared = rstride == 0;
  const int64_t Mp = round_up(M, 32), Np = round_up(N, 32);
  const RouteWs w = route_ws(ws, kind, dtype, B, H, N, M, D, shared);
  if (ws_bytes < w.bytes)
    return fail(FLAREPP_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, w.bytes);
  const float qscale = route_qscale(D);
  const int64_t rtHS = Mp * D, rtBS = shared ? 0 : H * Mp * D;
  const int64_t tokHS = N * D, tokBS = H * N * D;
  RoutePrepParams rp{};
  rp.src_bstride = rstride; rp.B = shared ? 1 : (int)B; rp.H = (int)H; rp.M = (int)M; rp.Mp = (int)Mp;
  rp.D = (int)D; rp.qscale = qscale;
  if (kind == FLAREPP_ENCODE) {
    rp.src = q; rp.q_op = w.q_op; rp.z_op = nullptr;
    HIPTRY((launch_route_prep<float, T>(rp, s)));
    DmajorParams dp{};
    dp.src = v; dp.dst = w.Vdm; dp.BH = B * H; dp.N = (int)N; dp.Np = (int)Np; dp.D = (int)D;
    HIPTRY(launch_dmajor<T>(dp, s));
    const EncPlan e = encode_plan(B, H, N, Mp, D);
    RouteParams r = encode_params(e, B, H, N, Mp, D);
    r.ka = k; r.ka_sb = tokBS; r.ka_sh = tokHS; r.ka_rows = (int)N;
    r.va = w.Vdm; r.va_sb = H * D * Np; r.va_sh = D * Np; r.va_ld = (int)Np;
    r.qs = w.q_op; r.qs_sb = rtBS; r.qs_sh = rtHS; r.qs_rows = (int)Mp;
    r.part_ml = w.part_ml; r.part_acc = w.part_acc;
    HIPTRY(launch_route<T>(r, (int)D, false, s));
    CombineParams c{};
    c.part_ml = w.part_ml; c.part_acc = w.part_acc; c.BH = B * H; c.R = e.nchunks; c.M = (int)M;
    c.Mp = (int)Mp; c.D = (int)D; c.qscale = qscale; c.out32 = (float*)out; c.lse = lse;
    HIPTRY(launch_combine_par<T>(c, s));
  } else {
    rp.src = k; rp.q_op = w.q_op; rp.z_op = nullptr;
    HIPTRY((launch_route_prep<float, T>(rp, s)));
    rp.src = v; rp.q_op = nullptr; rp.z_op = w.z_op;
    HIPTRY((launch_route_prep<float, T>(rp, s)));
    RouteParams r = decode_params(B, H, N, M, D);
    r.ka = w.q_op; r.ka_sb = rtBS; r.ka_sh = rtHS; r.ka_rows = (int)Mp;
    r.va = w.z_op; r.va_sb = shared ? 0 : H * D * Mp; r.va_sh = D * Mp; r.va_ld = (int)Mp;
    r.qs = q; r.qs_sb = tokBS; r.qs_sh = tokHS; r.qs_rows = (int)N;
    r.y = out; r.y_sb = N * H * D; r.y_row = H * D;
    HIPTRY(launch_route<T>(r, (int)D, true, s));
  }
  return ok();
}


// ---- backward (App. A.5) ----------------------------------------------------
// Work split of the SDPA backward over the long axis (keys of an encode,
// tokens of the decode): chunks per (b, h) and 32-position tiles per wave;
// and over the routes: a launch covers nsb route blocks (a window), sized so
// that four waves' route-gradient slots take at most 80 KB of LDS (two
// workgroups per CU); the windows run one after another.
struct BwdSplit {
  int waves, R, tpw, nsb;
};

BwdSplit bwd_split(int64_t BH, int64_t Nl, int D, int Mp, bool dec, int elem_bytes) {
  BwdSplit sp{};
  const int NS = Mp / 32;
  // LDS budget of a window at 4 waves: the CU's LDS split over as many
  // workgroups as the kernel's registers let run at once (bf16 at D = 16 fits
  // two waves per SIMD, so two workgroups of 80 KB; the other variants hold
  // one wave per SIMD, and a smaller window would only re-read the long side
  // once more per window).  FLAREPP_BWD_WINDOW_KB (testing and tuning)
  // overrides it.
  size_t budget = (D == 16 && elem_bytes == 2) ? 80 * 1024 : 160 * 1024;
  if (const char* f = std::getenv("FLAREPP_BWD_WINDOW_KB")) {
    const long kb = std::atol(f);
    if (kb >= 16 && kb <= 160) budget = (size_t)kb * 1024;
  }
  int nwin = 1;
  while (nwin < NS && flarepp::attn_bwd_lds_bytes(D, (int)cdiv(NS, nwin), Mp, dec, 4, elem_bytes) > budget)
    ++nwin;
  sp.nsb = (int)cdiv(NS, nwin);
  sp.waves = flarepp::attn_bwd_waves(D, sp.nsb, Mp, dec, elem_bytes);
  const int64_t tiles = cdiv(Nl, 32);
  int64_t R = std::max<int64_t>(1, std::min<int64_t>(cdiv(512, BH), cdiv(tiles, sp.waves)));
  const int64_t tpw = cdiv(tiles, R * sp.waves);
  R = cdiv(tiles, tpw * sp.waves);
  sp.R = (int)R;
  sp.tpw = (int)tpw;
  return sp;
}

// Split-K of the five token reductions dW = X^T dG, dW_O = Y^T dO (K = B N
// tokens), computed in one launch: about 512 workgroups in all (the GEMM's
// workgroup tile is 128 x 128 for C >= 128, else 64 x 64).
int gemm_splits(int64_t T, int64_t C, int* kchunk) {
  const int64_t tile = C >= 128 ? 128 : 64;
  const int64_t tiles = cdiv(C, tile) * cdiv(C, tile);
  int64_t splits = std::max<int64_t>(1, std::min<int64_t>(cdiv(T, 256), cdiv(512, 5 * tiles)));
  const int64_t kc = round_up(cdiv(T, splits), 64);
  *kchunk = (int)kc;
  return (int)cdiv(T, kc);
}

struct BwdWs {
  void *wf[4], *seeds_op, *K, *Kt, *Vdm, *Vtdm, *Y, *q_op, *z_op;
  void *fwf[2], *fq_op;  // fused encodes: W_K (key order), W_V fragments; Q(X) in q fragment order
  void *fwo, *fz_op;     // fused decode: W_O merge fragments, Z in z fragment order
  float* fqnorm2;        // fused decode: route-norm bounds of Q(X)
  float *part_ml, *part_acc, *Qf, *Zf, *L1, *L2, *L3;
  float *dZf, *dQf, *c1, *c2, *l1, *l2, *pa, *pg, *pq, *gpart;
  void *dY, *dK, *dV, *dKt, *dVt;
  void *dVlo, *dVtlo;  // bf16: the value gradients' low parts
  void *Qr, *Qt, *Zr, *dZr, *dZt, *dQr, *dQt, *Sr, *St;
  BwdSplit dec, enc;
  int splits, kchunk;
  size_t bytes;
};

// bf16: the encoders' value gradients (dV, dV~) are kept as bf16 pairs
// hi + lo between the SDPA backward and the weight-gradient GEMMs.  A value
// gradient P^T dOut over a near-uniform softmax is a common part (about the
// mean of dOut over the routes) plus a small token-dependent part, which
// falls below the bf16 step of the common part at large N; the weight
// gradient X^T dV is made of exactly that part (with hi alone dW_V at 2^20
// tokens is off by ~10% of its largest entry).  The key gradients
// dK = s dS^T Q have no common part (dS sums to zero over the routes).
// FLAREPP_BWD_NO_LO=1 (testing and tuning) keeps hi alone.
bool bwd_lo_parts(int dtype) {
  if (dtype != FLAREPP_BF16) return false;
  const char* f = std::getenv("FLAREPP_BWD_NO_LO");
  return !(f && std::atoi(f) != 0);
}

// The backward's forward runs its three calls on the fused kernels (which
// project inside the routing kernel) when the fused path covers the shape:
// the decode also writes Y and the per-token log-normaliser; K, V, K~, V~
// are still materialised for the reverse pass.
bool bwd_fused_encodes(int dtype, const MixerPlan& pl) { return pl.fused && dtype == FLAREPP_BF16; }

BwdWs bwd_ws(void* base, int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  const int64_t D = C / H, Mp = round_up(M, 32), Np = round_up(N, 32), DB = cdiv(D, 32);
  const size_t bs = dtype_bytes(dtype), f4 = sizeof(float);
  const int64_t T = B * N, BH = B * H;
  const EncPlan e = encode_plan(B, H, N, Mp, D);
  Carver cv(base);
  BwdWs w{};
  for (int i = 0; i < 4; ++i) w.wf[i] = cv.take(bs * C * C);
  w.seeds_op = cv.take(bs * H * Mp * D);
  w.K = cv.take(bs * BH * N * D);
  w.Kt = cv.take(bs * BH * N * D);
  w.Vdm = cv.take(bs * BH * D * Np);
  w.Vtdm = cv.take(bs * BH * D * Np);
  w.Y = cv.take(bs * T * C);
  w.q_op = cv.take(bs * BH * Mp * D);
  w.z_op = cv.take(bs * BH * D * Mp);
  // the encodes' partials: the unfused route's chunks or the fused encode's
  const MixerPlan pl = mixer_plan(dtype, B, N, C, H, M);
  const bool fused = bwd_fused_encodes(dtype, pl);
  const int64_t Rp = std::max<int64_t>(e.nchunks, fused ? pl.nchunks : 1);
  if (fused) {
    w.fwf[0] = cv.take(bs * C * C);
    w.fwf[1] = cv.take(bs * C * C);
    w.fq_op = cv.take(bs * BH * Mp * D);
    w.fwo = cv.take(bs * C * C);
    w.fz_op = cv.take(bs * BH * flarepp::z_frag_elems_per_head((int)Mp, (int)D));
    w.fqnorm2 = (float*)cv.take(f4 * BH * (Mp / 4));
  }
  w.part_ml = (float*)cv.take(f4 * Rp * BH * Mp * 2);
  w.part_acc = (float*)cv.take(f4 * Rp * BH * Mp * D);
  w.Qf = (float*)cv.take(f4 * BH * M * D);
  w.Zf = (float*)cv.take(f4 * BH * M * D);
  w.L1 = (float*)cv.take(f4 * BH * M);
  w.L2 = (float*)cv.take(f4 * BH * M);
  w.L3 = (float*)cv.take(f4 * BH * N);
  w.dY = cv.take(bs * T * C);
  w.dK = cv.take(bs * T * C);
  w.dV = cv.take(bs * T * C);
  w.dKt = cv.take(bs * T * C);
  w.dVt = cv.take(bs * T * C);
  if (bwd_lo_parts(dtype)) {
    w.dVlo = cv.take(bs * T * C);
    w.dVtlo = cv.take(bs * T * C);
  }
  w.dZf = (float*)cv.take(f4 * BH * M * D);
  w.dQf = (float*)cv.take(f4 * BH * M * D);
  w.c1 = (float*)cv.take(f4 * BH * Mp);
  w.c2 = (float*)cv.take(f4 * BH * Mp);
  w.l1 = (float*)cv.take(f4 * BH * Mp);
  w.l2 = (float*)cv.take(f4 * BH * Mp);
  w.Qr = cv.take(bs * BH * Mp * D);
  w.Qt = cv.take(bs * BH * Mp * 32 * DB);
  w.Zr = cv.take(bs * BH * Mp * D);
  w.dZr = cv.take(bs * BH * Mp * D);
  w.dZt = cv.take(bs * BH * Mp * 32 * DB);
  w.dQr = cv.take(bs * BH * Mp * D);
  w.dQt = cv.take(bs * BH * Mp * 32 * DB);
  w.Sr = cv.take(bs * H * Mp * D);
  w.St = cv.take(bs * H * Mp * 32 * DB);
  w.dec = bwd_split(BH, N, (int)D, (int)Mp, true, (int)bs);
  w.enc = bwd_split(BH, N, (int)D, (int)Mp, false, (int)bs);
  const int64_t R = std::max<int64_t>(std::max(w.dec.R, w.enc.R), 1);
  w.pa = (float*)cv.take(f4 * BH * R * Mp * D);
  w.pg = (float*)cv.take(f4 * BH * R * Mp * D);
  w.pq = (float*)cv.take(f4 * BH * R * Mp * D);
  w.splits = gemm_splits(T, C, &w.kchunk);
  w.gpart = (float*)cv.take(f4 * 5 * w.splits * C * C);
  w.bytes = cv.off;
  return w;
}

int check_backward_shape(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  TRY(check_mixer_shape(dtype, B, N, C, H, M));
  if (B * N > (int64_t(1) << 30)) return fail(FLAREPP_ERR_UNSUPPORTED, "B*N too large for the backward");
  return FLAREPP_OK;
}

// What backward_impl runs: the forward again and the reverse pass; the
// forward alone, keeping its statistics in the workspace and writing O (the
// training forward); or the reverse pass alone, on the statistics a training
// forward left in the workspace.
enum BwdMode { kBwdFull = 0, kBwdForward = 1, kBwdReverse = 2 };

// The mixer's reverse pass: the forward again (unfused kernels, which keep
// K, V, K~, V~, Y and the log-normalisers of both encodes), then the merge,
// call 3, call 2, call 1 and the projections in reverse order.
template <typename T>
int backward_impl(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M, const void* X,
                  const void* Wk, const void* Wv, const void* Wkt, const void* Wvt, const void* Wo,
                  const void* seeds, const void* dO, float* dX, float* dWk, float* dWv, float* dWkt,
                  float* dWvt, float* dWo, float* dseeds, float* dZ_out, float* dQ_out, void* ws,
                  size_t ws_bytes, hipStream_t s, int mode = kBwdFull, void* O = nullptr) {
  using namespace flarepp;
  const int64_t D = C / H, Mp = round_up(M, 32), Np = round_up(N, 32), DB = cdiv(D, 32);
  const int64_t NT = B * N, BH = B * H;
  const BwdWs w = bwd_ws(ws, dtype, B, N, C, H, M);
  if (ws_bytes < w.bytes)
    return fail(FLAREPP_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, w.bytes);
  const float qscale = route_qscale(D);
  const float sc = (float)(1.0 / std::sqrt((double)D));
  const bool f32 = std::is_same<T, float>::value;

  const void* w_in[4] = {Wk, Wv, Wkt, Wvt};
  const EncPlan e = encode_plan(B, H, N, Mp, D);
  const int64_t tokHS = N * D, tokBS = H * N * D, dmHS = D * Np, dmBS = H * D * Np;
  const int64_t rtHS = Mp * D, rtBS = H * Mp * D;

  // ---- forward with its statistics (kept in the workspace) ----
  if (mode != kBwdReverse) {
  WeightFragParams wp{};
  wp.C = (int)C;
  for (int i = 0; i < 4; ++i) { wp.w[i] = w_in[i]; wp.out[i] = w.wf[i]; }
  wp.nw = 4;
  HIPTRY(launch_weight_frags<T>(wp, s));
  ProjParams pp{};
  pp.x = X; pp.B = (int)B; pp.N = (int)N; pp.Np = (int)Np; pp.C = (int)C; pp.H = (int)H; pp.D = (int)D;
  pp.nw = 4;
  pp.wf[0] = w.wf[0]; pp.out[0] = w.K;    pp.layout[0] = kHeadsTokenMajor;
  pp.wf[1] = w.wf[1]; pp.out[1] = w.Vdm;  pp.layout[1] = kHeadsDMajor;
  pp.wf[2] = w.wf[2]; pp.out[2] = w.Kt;   pp.layout[2] = kHeadsTokenMajor;
  pp.wf[3] = w.wf[3]; pp.out[3] = w.Vtdm; pp.layout[3] = kHeadsDMajor;
  HIPTRY(launch_project<T>(pp, s));
  const MixerPlan pl = mixer_plan(dtype, B, N, C, H, M);
  // call 3 on the unfused decode (route operands as rows of Q(X) scaled and
  // Z d-major), which writes Y and the per-token log-normaliser
  auto unfused_call3 = [&]() -> int {
    RouteParams r3 = decode_params(B, H, N, M, D);
    r3.ka = w.q_op; r3.ka_sb = rtBS; r3.ka_sh = rtHS; r3.ka_rows = (int)Mp;
    r3.va = w.z_op; r3.va_sb = H * D * Mp; r3.va_sh = D * Mp; r3.va_ld = (int)Mp;
    r3.qs = w.K; r3.qs_sb = tokBS; r3.qs_sh = tokHS; r3.qs_rows = (int)N;
    r3.y = w.Y; r3.y_sb = N * C; r3.y_row = C; r3.lse2 = w.L3;
    HIPTRY(launch_route<T>(r3, (int)D, true, s));
    return FLAREPP_OK;
  };
  if (bwd_fused_encodes(dtype, pl)) {
    // calls 1 and 2 on the fused encodes, as in the forward.  Call 3 on the
    // fused decode where it has the per-group stages (C <= 128; the first
    // combine then also writes W_O's merge fragments): it writes Y and the
    // per-token log-normaliser for the reverse pass, and O (the training
    // forward's output; otherwise into dY's buffer, which the merge gradient
    // overwrites).  At C = 256 the unfused decode is the faster one here (no
    // projection or merge to repeat): the combines write its route operands.
    const int dkind = decode_kind_for((int)C, (int)D, (int)Mp, (int)dtype_bytes(dtype));
    const bool fdec = dkind != kDecodeStaged;
    PrepFusedParams fp{};
    fp.C = (int)C;
    fp.w[0] = Wk; fp.wf[0] = w.fwf[0]; fp.mode[0] = kFragKeyPerm;
    fp.w[1] = Wv; fp.wf[1] = w.fwf[1]; fp.mode[1] = kFragPlain;
    fp.w[2] = Wo; fp.wf[2] = w.fwo; fp.mode[2] = dkind == kDecodeStaged ? kFragMerge : kFragMergeHg;
    fp.nw = fdec ? 3 : 2;
    fp.seeds = seeds; fp.H = (int)H; fp.M = (int)M; fp.Mp = (int)Mp; fp.D = (int)D; fp.qscale = qscale;
    EncFusedParams ep{};
    ep.x = X; ep.wk_raw = Wkt; ep.wv_raw = Wvt; ep.seeds_raw = seeds;
    ep.q_sb = 0; ep.M = (int)M; ep.qscale = qscale;
    ep.B = (int)B; ep.N = (int)N; ep.C = (int)C; ep.H = (int)H; ep.Mp = (int)Mp; ep.QB = (int)(Mp / 32);
    ep.nqw = pl.nqw; ep.qgroups = pl.qgroups; ep.chunk = pl.chunk; ep.nchunks = pl.nchunks;
    ep.fast_lim = fast_limit(); ep.part_ml = w.part_ml; ep.part_acc = w.part_acc;
    HIPTRY(launch_encode_fused<T>(ep, (int)D, pl.waves, s));
    CombineParams cp{};
    cp.part_ml = w.part_ml; cp.part_acc = w.part_acc; cp.BH = BH; cp.R = pl.nchunks;
    cp.M = (int)M; cp.Mp = (int)Mp; cp.D = (int)D; cp.qscale = qscale; cp.frag = 1;
    cp.out32 = w.Qf; cp.lse = w.L1; cp.q_op = w.fq_op;
    cp.qnorm2 = fdec ? w.fqnorm2 : nullptr; cp.q_rows = fdec ? nullptr : w.q_op;
    cp.prep = fp; cp.prep_n = prep_fused_items(fp);
    HIPTRY(launch_combine_par<T>(cp, s));
    ep.wk_raw = ep.wv_raw = ep.seeds_raw = nullptr;
    ep.wkf = w.fwf[0]; ep.wvf = w.fwf[1]; ep.q_op = w.fq_op; ep.q_sb = H * Mp * D;
    HIPTRY(launch_encode_fused<T>(ep, (int)D, pl.waves, s));
    cp.out32 = w.Zf; cp.lse = w.L2; cp.q_op = nullptr; cp.qnorm2 = nullptr; cp.q_rows = nullptr;
    cp.z_op = fdec ? w.fz_op : nullptr; cp.z_rows = fdec ? nullptr : w.z_op;
    cp.prep_n = 0;
    HIPTRY(launch_combine_par<T>(cp, s));
    if (!fdec) {
      TRY(unfused_call3());
    } else {
    DecFusedParams dp{};
    dp.x = X; dp.wkf = w.fwf[0]; dp.wof = w.fwo; dp.q_op = w.fq_op; dp.z_op = w.fz_op; dp.qnorm2 = w.fqnorm2;
    dp.B = (int)B; dp.N = (int)N; dp.C = (int)C; dp.H = (int)H; dp.M = (int)M; dp.Mp = (int)Mp;
    dp.fast_lim = fast_limit(); dp.y = w.Y; dp.lse2 = w.L3;
    dp.o = mode == kBwdForward ? O : w.dY; dp.res = nullptr;
    dp.stage_elems = decode_stage_elems((int)C, (int)D, (int)Mp);
    dp.stage_bytes = (int)(dkind == kDecodePersist ? persist_stage_bytes((int)D, (int)Mp, (int)dtype_bytes(dtype))
                                                   : dec2_stage_bytes((int)C, (int)D, (int)Mp, (int)dtype_bytes(dtype)));
    dp.kind = dkind;
    HIPTRY(launch_decode_fused<T>(dp, (int)D, s));
    if (mode == kBwdForward) return ok();
    }
  } else {
  RoutePrepParams sp{};
  sp.src = seeds; sp.src_bstride = 0; sp.B = 1; sp.H = (int)H; sp.M = (int)M; sp.Mp = (int)Mp;
  sp.D = (int)D; sp.qscale = qscale; sp.q_op = w.seeds_op; sp.z_op = nullptr;
  HIPTRY((launch_route_prep<T, T>(sp, s)));
  RouteParams r1 = encode_params(e, B, H, N, Mp, D);
  r1.ka = w.Kt; r1.ka_sb = tokBS; r1.ka_sh = tokHS; r1.ka_rows = (int)N;
  r1.va = w.Vtdm; r1.va_sb = dmBS; r1.va_sh = dmHS; r1.va_ld = (int)Np;
  r1.qs = w.seeds_op; r1.qs_sb = 0; r1.qs_sh = rtHS; r1.qs_rows = (int)Mp;
  r1.part_ml = w.part_ml; r1.part_acc = w.part_acc;
  HIPTRY(launch_route<T>(r1, (int)D, false, s));
  CombineParams c1{};
  c1.part_ml = w.part_ml; c1.part_acc = w.part_acc; c1.BH = BH; c1.R = e.nchunks;
  c1.M = (int)M; c1.Mp = (int)Mp; c1.D = (int)D; c1.qscale = qscale;
  c1.out32 = w.Qf; c1.lse = w.L1; c1.q_op = w.q_op; c1.z_op = nullptr;
  HIPTRY(launch_combine_par<T>(c1, s));
  RouteParams r2 = r1;
  r2.ka = w.K; r2.va = w.Vdm;
  r2.qs = w.q_op; r2.qs_sb = rtBS; r2.qs_sh = rtHS; r2.qs_rows = (int)Mp;
  HIPTRY(launch_route<T>(r2, (int)D, false, s));
  CombineParams c2 = c1;
  c2.out32 = w.Zf; c2.lse = w.L2; c2.q_op = nullptr; c2.z_op = w.z_op;
  HIPTRY(launch_combine_par<T>(c2, s));
  TRY(unfused_call3());
  }
  }
  if (mode == kBwdForward) {  // the training forward's output O = Y W_O (the fused decode returned above)
    GemmParams go{};
    go.M = (int)NT; go.N = (int)C; go.K = (int)C; go.nseg = 1; go.nprob = 1; go.splits = 1;
    go.a[0] = w.Y; go.a_m = C; go.a_k = 1;
    go.b[0] = Wo; go.b_k = C; go.b_n = 1;
    go.kchunk = (int)round_up(C, 64); go.c = O; go.c_t = 1; go.ldc = C; go.split_stride = 0;
    HIPTRY(launch_gemm<T>(go, s));
    return ok();
  }

  // ---- merge: dY = dO W_O^T (dW_O is computed with the weight gradients) ----
  GemmParams g{};
  g.M = (int)NT; g.N = (int)C; g.K = (int)C; g.nseg = 1; g.nprob = 1; g.splits = 1;
  g.a[0] = dO; g.a_m = C; g.a_k = 1;
  g.b[0] = Wo; g.b_k = 1; g.b_n = C;
  g.kchunk = (int)round_up(C, 64); g.c = w.dY; g.c_t = 1; g.ldc = C; g.split_stride = 0;
  HIPTRY(launch_gemm<T>(g, s));

  // one SDPA backward, launched once per window of route blocks; the later
  // windows add to the long-side gradients of the earlier ones
  auto attn_windows = [&](const AttnBwdParams& a, const BwdSplit& sp, bool dec) -> int {
    const int NS = (int)(Mp / 32);
    for (int w0 = 0; w0 < NS; w0 += sp.nsb) {
      AttnBwdParams q = a;
      q.sb0 = w0;
      q.nsb = std::min(sp.nsb, NS - w0);
      if (w0 > 0) q.acc_b = q.acc_g = 1;
      HIPTRY(launch_attn_bwd<T>(q, (int)D, dec, s));
    }
    return FLAREPP_OK;
  };

  // ---- route-side operands of the calls: Q (rows and transposed), Z rows,
  // the seeds (rows and transposed) ----
  BwdPrepParams bp{};
  bp.M = (int)M; bp.Mp = (int)Mp; bp.D = (int)D; bp.njobs = 3;
  bp.job[0].src = w.Qf; bp.job[0].src_is_f32 = 1; bp.job[0].O = (int)BH;
  bp.job[0].rows = w.Qr; bp.job[0].tfrag = w.Qt; bp.job[0].rows_scale = sc * 1.4426950408889634f;
  bp.job[1].src = w.Zf; bp.job[1].src_is_f32 = 1; bp.job[1].O = (int)BH; bp.job[1].rows = w.Zr;
  bp.job[2].src = seeds; bp.job[2].src_is_f32 = f32 ? 1 : 0; bp.job[2].O = (int)H;
  bp.job[2].rows = w.Sr; bp.job[2].tfrag = w.St; bp.job[2].rows_scale = sc * 1.4426950408889634f;
  HIPTRY(launch_bwd_prep<T>(bp, s));

  // ---- call 3 (decode): queries K, keys Q, values Z ----
  const int64_t tfS = Mp * 32 * DB;  // elements per head of a transposed-fragment operand
  AttnBwdParams a3{};
  a3.B = (int)B; a3.H = (int)H; a3.Nl = (int)N; a3.M = (int)M; a3.Mp = (int)Mp;
  a3.R = w.dec.R; a3.tpw = w.dec.tpw; a3.s = sc; a3.sl2 = sc * 1.4426950408889634f;
  a3.ash = w.Qr; a3.ash_sb = rtBS; a3.ash_sh = rtHS;
  a3.asht = w.Qt; a3.asht_sb = H * tfS; a3.asht_sh = tfS;
  a3.gsh = w.Zr; a3.gsh_sb = rtBS; a3.gsh_sh = rtHS;
  a3.blo = w.K; a3.blo_sb = tokBS; a3.blo_sh = tokHS; a3.blo_sn = D; a3.blo_sd = 1;
  a3.glo = w.dY; a3.glo_sb = N * C; a3.glo_sh = D; a3.glo_sn = C; a3.glo_sd = 1;
  a3.ylo = w.Y; a3.ylo_sb = N * C; a3.ylo_sh = D; a3.ylo_sn = C; a3.lcol = w.L3;
  a3.dout_b = w.dK; a3.acc_b = 0;
  a3.part_a = w.pa; a3.part_g = w.pg;
  TRY(attn_windows(a3, w.dec, true));

  // ---- call 2 (encode): queries Q, keys K, values V; dOut = dZ, the sum of
  // the decode's partials ----
  BwdReduceParams rd{};
  rd.P = 1; rd.O = (int)BH; rd.M = (int)M; rd.Mp = (int)Mp; rd.D = (int)D;
  rd.part0 = w.pg; rd.R0 = w.dec.R; rd.out = dZ_out ? dZ_out : w.dZf;
  HIPTRY(launch_bwd_reduce(rd, s));
  bp = BwdPrepParams{};
  bp.M = (int)M; bp.Mp = (int)Mp; bp.D = (int)D; bp.njobs = 1;
  bp.job[0].src = rd.out; bp.job[0].src_is_f32 = 1; bp.job[0].O = (int)BH;
  bp.job[0].rows = w.dZr; bp.job[0].tfrag = w.dZt; bp.job[0].dot = w.Zf; bp.job[0].c = w.c2;
  bp.job[0].lse = w.L2; bp.job[0].l2 = w.l2;
  HIPTRY(launch_bwd_prep<T>(bp, s));
  AttnBwdParams a2{};
  a2.B = (int)B; a2.H = (int)H; a2.Nl = (int)N; a2.M = (int)M; a2.Mp = (int)Mp;
  a2.R = w.enc.R; a2.tpw = w.enc.tpw; a2.s = sc; a2.sl2 = a3.sl2;
  a2.ash = w.Qr; a2.ash_sb = rtBS; a2.ash_sh = rtHS;
  a2.asht = w.Qt; a2.asht_sb = H * tfS; a2.asht_sh = tfS;
  a2.gsh = w.dZr; a2.gsh_sb = rtBS; a2.gsh_sh = rtHS;
  a2.gsht = w.dZt; a2.gsht_sb = H * tfS; a2.gsht_sh = tfS;
  a2.lrow = w.l2; a2.crow = w.c2;
  a2.blo = w.K; a2.blo_sb = tokBS; a2.blo_sh = tokHS; a2.blo_sn = D; a2.blo_sd = 1;
  a2.glo = w.Vdm; a2.glo_sb = dmBS; a2.glo_sh = dmHS; a2.glo_sn = 1; a2.glo_sd = Np;
  a2.dout_b = w.dK; a2.acc_b = 1; a2.dout_g = w.dV; a2.dout_g_lo = w.dVlo;
  a2.part_a = w.pq;
  TRY(attn_windows(a2, w.enc, false));

  // ---- call 1 (query synthesis): queries = seeds (shared), keys K~, values
  // V~; dOut = dQ, the decode's and the encode's shares summed ----
  rd.part0 = w.pa; rd.R0 = w.dec.R; rd.part1 = w.pq; rd.R1 = w.enc.R; rd.out = dQ_out ? dQ_out : w.dQf;
  HIPTRY(launch_bwd_reduce(rd, s));
  bp = BwdPrepParams{};
  bp.M = (int)M; bp.Mp = (int)Mp; bp.D = (int)D; bp.njobs = 1;
  bp.job[0].src = rd.out; bp.job[0].src_is_f32 = 1; bp.job[0].O = (int)BH;
  bp.job[0].rows = w.dQr; bp.job[0].tfrag = w.dQt; bp.job[0].dot = w.Qf; bp.job[0].c = w.c1;
  bp.job[0].lse = w.L1; bp.job[0].l2 = w.l1;
  HIPTRY(launch_bwd_prep<T>(bp, s));
  AttnBwdParams a1 = a2;
  a1.ash = w.Sr; a1.ash_sb = 0; a1.ash_sh = rtHS;
  a1.asht = w.St; a1.asht_sb = 0; a1.asht_sh = tfS;
  a1.gsh = w.dQr; a1.gsht = w.dQt;
  a1.lrow = w.l1; a1.crow = w.c1;
  a1.blo = w.Kt; a1.glo = w.Vtdm;
  a1.dout_b = w.dKt; a1.acc_b = 0; a1.dout_g = w.dVt; a1.dout_g_lo = w.dVtlo;
  a1.part_a = w.pa;
  TRY(attn_windows(a1, w.enc, false));
  rd = BwdReduceParams{};
  rd.P = (int)B; rd.O = (int)H; rd.M = (int)M; rd.Mp = (int)Mp; rd.D = (int)D;
  rd.part0 = w.pa; rd.R0 = w.enc.R; rd.out = dseeds;
  HIPTRY(launch_bwd_reduce(rd, s));

  // ---- projections: dX = sum_j dG_j W_j^T; the weight gradients
  // dW_j = X^T dG_j and dW_O = Y^T dO in one split-K launch ----
  GemmParams gx{};
  gx.M = (int)NT; gx.N = (int)C; gx.K = (int)C; gx.nseg = 4; gx.nprob = 1; gx.splits = 1;
  const void* G[4] = {w.dK, w.dV, w.dKt, w.dVt};
  for (int j = 0; j < 4; ++j) { gx.a[j] = G[j]; gx.b[j] = w_in[j]; }
  gx.a_m = C; gx.a_k = 1; gx.b_k = 1; gx.b_n = C;
  gx.kchunk = (int)round_up(C, 64); gx.c = dX; gx.c_t = 0; gx.ldc = C; gx.split_stride = 0;
  HIPTRY(launch_gemm<T>(gx, s));
  GemmParams gw{};
  gw.M = (int)C; gw.N = (int)C; gw.K = (int)NT; gw.nseg = 1; gw.nprob = 5; gw.splits = w.splits;
  const void* wa[5] = {X, X, X, X, w.Y};
  const void* wb[5] = {w.dK, w.dV, w.dKt, w.dVt, dO};
  for (int j = 0; j < 5; ++j) { gw.a[j] = wa[j]; gw.b[j] = wb[j]; }
  gw.a_m = 1; gw.a_k = C; gw.b_k = C; gw.b_n = 1;
  gw.kchunk = w.kchunk; gw.c = w.gpart; gw.c_t = 0; gw.ldc = C; gw.split_stride = C * C;
  if (!dWkt) {
    // tied weights (W~_K = W_K, W~_V = W_V): dW_K = X^T (dK + dK~) and
    // dW_V = X^T (dV + dV~) (with the low parts under bf16), each one problem
    // over K segments; then dW_O
    const void* seg[3][4] = {{w.dK, w.dKt, nullptr, nullptr},
                             {w.dV, w.dVt, w.dVlo, w.dVtlo},
                             {dO, nullptr, nullptr, nullptr}};
    const void* sa[3] = {X, X, w.Y};
    gw.nprob = 3; gw.nseg = 4;
    for (int j = 0; j < 3; ++j)
      for (int k = 0; k < 4; ++k) { gw.a[4 * j + k] = sa[j]; gw.b[4 * j + k] = seg[j][k]; }
    HIPTRY(launch_gemm<T>(gw, s));
    float* dW3[3] = {dWk, dWv, dWo};
    HIPTRY(launch_sum_splits(w.gpart, dW3, C * C, w.splits, 3, s));
    return ok();
  }
  if (w.dVlo) {
    // dW_V and dW~_V as X^T hi + X^T lo (two K segments); the other three
    // problems have one (a null second segment)
    const void* lo[5] = {nullptr, w.dVlo, nullptr, w.dVtlo, nullptr};
    gw.nseg = 2;
    for (int j = 0; j < 5; ++j) {
      gw.a[2 * j] = gw.a[2 * j + 1] = wa[j];
      gw.b[2 * j] = wb[j];
      gw.b[2 * j + 1] = lo[j];
    }
  }
  HIPTRY(launch_gemm<T>(gw, s));
  float* dW[5] = {dWk, dWv, dWkt, dWvt, dWo};
  HIPTRY(launch_sum_splits(w.gpart, dW, C * C, w.splits, 5, s));
  return ok();
}

int backward_entry(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M, const void* X,
                   const void* Wk, const void* Wv, const void* Wkt, const void* Wvt, const void* Wo,
                   const void* seeds, const void* dO, float* dX, float* dWk, float* dWv, float* dWkt,
                   float* dWvt, float* dWo, float* dseeds, float* dZ_out, float* dQ_out, void* ws,
                   size_t ws_bytes, void* stream, bool shared = false, int mode = kBwdFull) {
  TRY(check_backward_shape(dtype, B, N, C, H, M));
  if (shared) dWkt = dWvt = nullptr;
  const void* in[] = {X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO};
  const char* in_names[] = {"X", "Wk", "Wv", "Wkt", "Wvt", "Wo", "seeds", "dO"};
  for (int i = 0; i < 8; ++i) TRY(check_ptr(in[i], in_names[i]));
  // shared: the tied weights' gradients land in dWk and dWv (dWkt, dWvt null)
  const float* out[] = {dX, dWk, dWv, dWkt, dWvt, dWo, dseeds};
  const char* out_names[] = {"dX", "dWk", "dWv", "dWkt", "dWvt", "dWo", "dseeds"};
  for (int i = 0; i < 7; ++i)
    if (!(shared && (i == 3 || i == 4))) TRY(check_ptr(out[i], out_names[i]));
  TRY(check_ptr(dZ_out, "dZ_out", true));
  TRY(check_ptr(dQ_out, "dQ_out", true));
  if (!ws) return fail(FLAREPP_ERR_WORKSPACE, "workspace is NULL");
  TRY(check_ptr(ws, "ws"));
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == FLAREPP_F32)
    return backward_impl<float>(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, dX, dWk, dWv, dWkt,
                                dWvt, dWo, dseeds, dZ_out, dQ_out, ws, ws_bytes, s, mode);
  return backward_impl<__bf16>(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, dX, dWk, dWv, dWkt,
                               dWvt, dWo, dseeds, dZ_out, dQ_out, ws, ws_bytes, s, mode);
}

int forward_train_entry(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M, const void* X,
                        const void* Wk, const void* Wv, const void* Wkt, const void* Wvt, const void* Wo,
                        const void* seeds, void* O, void* ws, size_t ws_bytes, void* stream) {
  TRY(check_backward_shape(dtype, B, N, C, H, M));
  const void* in[] = {X, Wk, Wv, Wkt, Wvt, Wo, seeds, O};
  const char* in_names[] = {"X", "Wk", "Wv", "Wkt", "Wvt", "Wo", "seeds", "O"};
  for (int i = 0; i < 8; ++i) TRY(check_ptr(in[i], in_names[i]));
  if (!ws) return fail(FLAREPP_ERR_WORKSPACE, "workspace is NULL");
  TRY(check_ptr(ws, "ws"));
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == FLAREPP_F32)
    return backward_impl<float>(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, nullptr, nullptr, nullptr,
                                nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, ws, ws_bytes, s,
                                kBwdForward, O);
  return backward_impl<__bf16>(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, nullptr, nullptr, nullptr,
                               nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, ws, ws_bytes, s,
                               kBwdForward, O);
}

// ---- allocation-free variant of the mixer forward ----------------------------
// The workspace of flarepp_mixer_forward_noalloc is this file-scope device
// array: every device the library runs on holds its own copy until the
// process ends.  In host code the name is only a host-side stand-in; kernels
// get the device address that hipGetSymbolAddress returns for the current
// device, looked up once per device and kept in g_scratch.
constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxScratchDevices];

// The scratch array's address on device `dev` (the current device).
int scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(FLAREPP_ERR_UNSUPPORTED, "device %d is beyond the %d the library tracks", dev, kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(FLAREPP_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    // the runtime resolved the device copy: its size is the array's, and its
    // address is not the host-side stand-in
    size_t n = 0;
    e = hipGetSymbolSize(&n, HIP_SYMBOL(scratch));
    if (e != hipSuccess || n != kScratchBytes || p == static_cast<void*>(scratch))
      return fail(FLAREPP_ERR_HIP, "the scratch array did not resolve on device %d (%s, %zu bytes)", dev,
                  hipGetErrorString(e), n);
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return FLAREPP_OK;
}

}  // namespace

extern "C" {

const char* flarepp_last_error(void) { return g_last_error.c_str(); }

const char* flarepp_version(void) { return "flarepp 0.1 (gfx950)"; }

size_t flarepp_project_workspace_bytes(int dtype, int64_t C) {
  if (check_dtype(dtype) != FLAREPP_OK || C < 1 || C > kMaxWidth) return 0;
  return 4 * align256((size_t)dtype_bytes(dtype) * C * C);
}

int flarepp_project(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, const void* X,
                    const void* Wk, const void* Wv, const void* Wkt, const void* Wvt, void* K,
                    void* V, void* Kt, void* Vt, void* ws, size_t ws_bytes, void* stream) {
  TRY(check_mixer_shape(dtype, B, N, C, H, 1));
  TRY(check_ptr(X, "X"));
  const void* W[4] = {Wk, Wv, Wkt, Wvt};
  void* Out[4] = {K, V, Kt, Vt};
  const char* wn[4] = {"Wk", "Wv", "Wkt", "Wvt"};
  const char* on[4] = {"K", "V", "Kt", "Vt"};
  int n = 0;
  for (int i = 0; i < 4; ++i) {
    if (!W[i] != !Out[i])
      return fail(FLAREPP_ERR_INVALID_ARG, "%s and %s must both be given or both be NULL", wn[i], on[i]);
    if (W[i]) {
      TRY(check_ptr(W[i], wn[i]));
      TRY(check_ptr(Out[i], on[i]));
      ++n;
    }
  }
  if (n == 0) return fail(FLAREPP_ERR_INVALID_ARG, "no (weight, output) pair given");
  if (!ws) return fail(FLAREPP_ERR_WORKSPACE, "workspace is NULL");
  TRY(check_ptr(ws, "ws"));
  const size_t need = flarepp_project_workspace_bytes(dtype, C);
  if (ws_bytes < need)
    return fail(FLAREPP_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, need);
  using namespace flarepp;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t slot = align256((size_t)dtype_bytes(dtype) * C * C);
  WeightFragParams wp{};
  ProjParams pp{};
  wp.C = (int)C;
  pp.x = X; pp.B = (int)B; pp.N = (int)N; pp.Np = (int)round_up(N, 32); pp.C = (int)C;
  pp.H = (int)H; pp.D = (int)(C / H);
  for (int i = 0; i < 4; ++i) {
    if (!W[i]) continue;
    void* frag = static_cast<char*>(ws) + slot * wp.nw;
    wp.w[wp.nw] = W[i]; wp.out[wp.nw] = frag; ++wp.nw;
    pp.wf[pp.nw] = frag; pp.out[pp.nw] = Out[i]; pp.layout[pp.nw] = kHeadsTokenMajor; ++pp.nw;
  }
  if (dtype == FLAREPP_F32) {
    HIPTRY(launch_weight_frags<float>(wp, s));
    HIPTRY(launch_project<float>(pp, s));
  } else {
    HIPTRY(launch_weight_frags<__bf16>(wp, s));
    HIPTRY(launch_project<__bf16>(pp, s));
  }
  return ok();
}

size_t flarepp_route_workspace_bytes(int kind, int dtype, int64_t B, int64_t H, int64_t N, int64_t M,
                                     int64_t D) {
  if (check_route_shape(kind, dtype, B, H, N, M, D) != FLAREPP_OK) return 0;
  return route_ws(nullptr, kind, dtype, B, H, N, M, D, false).bytes;
}

int flarepp_route(int kind, int dtype, int64_t B, int64_t H, int64_t N, int64_t M, int64_t D,
                  const void* q, int64_t route_batch_stride, const void* k, const void* v, void* out,
                  float* lse, void* ws, size_t ws_bytes, void* stream) {
  TRY(check_route_shape(kind, dtype, B, H, N, M, D));
  if (route_batch_stride != 0 && route_batch_stride != H * M * D)
    return fail(FLAREPP_ERR_INVALID_ARG, "route_batch_stride=%lld must be 0 or H*M*D=%lld",
                (long long)route_batch_stride, (long long)(H * M * D));
  TRY(check_ptr(q, "q"));
  TRY(check_ptr(k, "k"));
  TRY(check_ptr(v, "v"));
  TRY(check_ptr(out, "out"));
  if (kind == FLAREPP_DECODE && lse) return fail(FLAREPP_ERR_INVALID_ARG, "lse must be NULL for DECODE");
  TRY(check_ptr(lse, "lse", true));
  if (!ws) return fail(FLAREPP_ERR_WORKSPACE, "workspace is NULL");
  TRY(check_ptr(ws, "ws"));
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == FLAREPP_F32)
    return route_impl<float>(kind, dtype, B, H, N, M, D, q, route_batch_stride, k, v, out, lse, ws,
                             ws_bytes, s);
  return route_impl<__bf16>(kind, dtype, B, H, N, M, D, q, route_batch_stride, k, v, out, lse, ws,
                            ws_bytes, s);
}

size_t flarepp_mixer_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  if (check_mixer_shape(dtype, B, N, C, H, M) != FLAREPP_OK) return 0;
  return mixer_ws(nullptr, dtype, B, N, C, H, M, mixer_plan(dtype, B, N, C, H, M)).bytes;
}

int flarepp_mixer_path(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  TRY(check_mixer_shape(dtype, B, N, C, H, M));
  return mixer_plan(dtype, B, N, C, H, M).fused ? FLAREPP_PATH_FUSED : FLAREPP_PATH_UNFUSED;
}

int flarepp_mixer_forward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                          const void* X, const void* Wk, const void* Wv, const void* Wkt,
                          const void* Wvt, const void* Wo, const void* seeds, void* O, void* ws,
                          size_t ws_bytes, void* stream) {
  return mixer_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, O, nullptr, nullptr,
                     nullptr, ws, ws_bytes, stream, nullptr, 0);
}

size_t flarepp_mixer_noalloc_max_bytes(void) { return kScratchBytes; }

int flarepp_mixer_forward_noalloc(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                  const void* X, const void* Wk, const void* Wv, const void* Wkt,
                                  const void* Wvt, const void* Wo, const void* seeds, void* O,
                                  void* stream) {
  TRY(check_mixer_shape(dtype, B, N, C, H, M));
  const MixerPlan pl = mixer_plan(dtype, B, N, C, H, M);
  if (!pl.fused)
    return fail(FLAREPP_ERR_UNSUPPORTED,
                "the allocation-free mixer runs the fused kernels only; this shape (C=%lld, H=%lld, M=%lld) takes "
                "the unfused path, whose workspace holds token-sized tensors",
                (long long)C, (long long)H, (long long)M);
  const size_t need = mixer_ws(nullptr, dtype, B, N, C, H, M, pl).bytes;
  if (need > kScratchBytes)
    return fail(FLAREPP_ERR_WORKSPACE,
                "this shape needs %zu bytes of workspace, more than the %zu of the allocation-free mixer's scratch array",
                need, kScratchBytes);
  int dev = -1;
  HIPTRY(hipGetDevice(&dev));
  if (stream) {
    hipDevice_t sdev = -1;
    HIPTRY(hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev));
    if (sdev != dev)
      return fail(FLAREPP_ERR_INVALID_ARG, "the stream belongs to device %d, the current device is %d", (int)sdev, dev);
  }
  void* ws = nullptr;
  TRY(scratch_address(dev, &ws));
  return mixer_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, O, nullptr, nullptr, nullptr, ws,
                     kScratchBytes, stream, nullptr, 0);
}

int flarepp_mixer_forward_profiled(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                   const void* X, const void* Wk, const void* Wv, const void* Wkt,
                                   const void* Wvt, const void* Wo, const void* seeds, void* O,
                                   void* ws, size_t ws_bytes, void* stream, void* const* events,
                                   int n_events) {
  return mixer_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, O, nullptr, nullptr,
                     nullptr, ws, ws_bytes, stream, events, n_events);
}

int flarepp_mixer_stage(int stage, int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                        const void* X, const void* Wk, const void* Wv, const void* Wkt,
                        const void* Wvt, const void* Wo, const void* seeds, void* O, void* ws,
                        size_t ws_bytes, void* stream) {
  if (stage < 1) return fail(FLAREPP_ERR_INVALID_ARG, "stage=%d must be in [1, %d]", stage, FLAREPP_PROFILE_EVENTS - 1);
  return mixer_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, O, nullptr, nullptr,
                     nullptr, ws, ws_bytes, stream, nullptr, 0, stage);
}

int flarepp_mixer_forward_debug(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                const void* X, const void* Wk, const void* Wv, const void* Wkt,
                                const void* Wvt, const void* Wo, const void* seeds, void* O,
                                float* Q_out, float* Z_out, void* Y_out, void* ws, size_t ws_bytes,
                                void* stream) {
  return mixer_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, O, Q_out, Z_out, Y_out,
                     ws, ws_bytes, stream, nullptr, 0);
}

size_t flarepp_flare_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  if (check_mixer_shape(dtype, B, N, C, H, M) != FLAREPP_OK) return 0;
  return mixer_ws(nullptr, dtype, B, N, C, H, M, mixer_plan(dtype, B, N, C, H, M), true).bytes;
}

int flarepp_flare_forward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                          const void* X, const void* Wk, const void* Wv, const void* Wo,
                          const void* queries, void* O, void* ws, size_t ws_bytes, void* stream) {
  return mixer_entry(dtype, B, N, C, H, M, X, Wk, Wv, nullptr, nullptr, Wo, queries, O, nullptr, nullptr,
                     nullptr, ws, ws_bytes, stream, nullptr, 0, 0, true);
}

int flarepp_flare_forward_debug(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                const void* X, const void* Wk, const void* Wv, const void* Wo,
                                const void* queries, void* O, float* Z_out, void* Y_out, void* ws,
                                size_t ws_bytes, void* stream) {
  return mixer_entry(dtype, B, N, C, H, M, X, Wk, Wv, nullptr, nullptr, Wo, queries, O, nullptr, Z_out,
                     Y_out, ws, ws_bytes, stream, nullptr, 0, 0, true);
}

size_t flarepp_block_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  if (check_mixer_shape(dtype, B, N, C, H, M) != FLAREPP_OK) return 0;
  return align256((size_t)dtype_bytes(dtype) * B * N * C) +
         mixer_ws(nullptr, dtype, B, N, C, H, M, mixer_plan(dtype, B, N, C, H, M)).bytes;
}

int flarepp_block_forward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M, const void* X,
                          const void* gamma, const void* beta, float eps, const void* Wk, const void* Wv,
                          const void* Wkt, const void* Wvt, const void* Wo, const void* seeds, void* O,
                          void* ws, size_t ws_bytes, void* stream) {
  TRY(check_mixer_shape(dtype, B, N, C, H, M));
  const void* in[] = {X, gamma, beta, Wk, Wv, Wkt, Wvt, Wo, seeds, O};
  const char* names[] = {"X", "gamma", "beta", "Wk", "Wv", "Wkt", "Wvt", "Wo", "seeds", "O"};
  for (int i = 0; i < 10; ++i) TRY(check_ptr(in[i], names[i]));
  if (!(eps > 0.f) || !std::isfinite(eps)) return fail(FLAREPP_ERR_INVALID_ARG, "eps=%g must be positive", (double)eps);
  if (O == X) return fail(FLAREPP_ERR_INVALID_ARG, "O must not alias X (X is read again for the residual)");
  if (!ws) return fail(FLAREPP_ERR_WORKSPACE, "workspace is NULL");
  TRY(check_ptr(ws, "ws"));
  const size_t xn_bytes = align256((size_t)dtype_bytes(dtype) * B * N * C);
  const size_t need = flarepp_block_workspace_bytes(dtype, B, N, C, H, M);
  if (ws_bytes < need)
    return fail(FLAREPP_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* Xn = ws;
  void* mws = static_cast<char*>(ws) + xn_bytes;
  flarepp::LayerNormParams lp{};
  lp.x = X; lp.gamma = gamma; lp.beta = beta; lp.y = Xn; lp.T = B * N; lp.C = (int)C; lp.eps = eps;
  if (dtype == FLAREPP_F32) {
    HIPTRY(flarepp::launch_layernorm<float>(lp, s));
    return mixer_impl<float>(dtype, B, N, C, H, M, Xn, Wk, Wv, Wkt, Wvt, Wo, seeds, O, nullptr, nullptr, nullptr,
                             mws, ws_bytes - xn_bytes, s, nullptr, 0, false, X);
  }
  HIPTRY(flarepp::launch_layernorm<__bf16>(lp, s));
  return mixer_impl<__bf16>(dtype, B, N, C, H, M, Xn, Wk, Wv, Wkt, Wvt, Wo, seeds, O, nullptr, nullptr, nullptr,
                            mws, ws_bytes - xn_bytes, s, nullptr, 0, false, X);
}

// Block backward workspace: the normalised tokens, their statistics, the
// mixer's input gradient (fp32), the dgamma / dbeta partials, then the mixer
// backward's own workspace.
struct BlockBwdWs {
  void *xn, *ws;
  float *mean, *rstd, *dxn, *part;
  int nchunks;
  int64_t chunk;
  size_t bytes, ws_bytes;
};

BlockBwdWs block_bwd_ws(void* base, int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  const int64_t T = B * N;
  Carver cv(base);
  BlockBwdWs w{};
  w.chunk = std::max<int64_t>(1, cdiv(T, 1024));
  w.nchunks = (int)cdiv(T, w.chunk);
  w.xn = cv.take((size_t)dtype_bytes(dtype) * T * C);
  w.mean = (float*)cv.take(sizeof(float) * T);
  w.rstd = (float*)cv.take(sizeof(float) * T);
  w.dxn = (float*)cv.take(sizeof(float) * T * C);
  w.part = (float*)cv.take(sizeof(float) * 2 * w.nchunks * C);
  w.ws_bytes = bwd_ws(nullptr, dtype, B, N, C, H, M).bytes;
  w.ws = cv.take(w.ws_bytes);
  w.bytes = cv.off;
  return w;
}

size_t flarepp_block_backward_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M) {
  if (check_backward_shape(dtype, B, N, C, H, M) != FLAREPP_OK) return 0;
  return block_bwd_ws(nullptr, dtype, B, N, C, H, M).bytes;
}

int flarepp_block_backward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M, const void* X,
                           const void* gamma, const void* beta, float eps, const void* Wk, const void* Wv,
                           const void* Wkt, const void* Wvt, const void* Wo, const void* seeds, const void* dO,
                           float* dX, float* dgamma, float* dbeta, float* dWk, float* dWv, float* dWkt,
                           float* dWvt, float* dWo, float* dseeds, void* ws, size_t ws_bytes, void* stream) {
  TRY(check_backward_shape(dtype, B, N, C, H, M));
  const void* in[] = {X, gamma, beta, Wk, Wv, Wkt, Wvt, Wo, seeds, dO};
  const char* in_names[] = {"X", "gamma", "beta", "Wk", "Wv", "Wkt", "Wvt", "Wo", "seeds", "dO"};
  for (int i = 0; i < 10; ++i) TRY(check_ptr(in[i], in_names[i]));
  const float* out[] = {dX, dgamma, dbeta, dWk, dWv, dWkt, dWvt, dWo, dseeds};
  const char* out_names[] = {"dX", "dgamma", "dbeta", "dWk", "dWv", "dWkt", "dWvt", "dWo", "dseeds"};
  for (int i = 0; i < 9; ++i) TRY(check_ptr(out[i], out_names[i]));
  if (!(eps > 0.f) || !std::isfinite(eps)) return fail(FLAREPP_ERR_INVALID_ARG, "eps=%g must be positive", (double)eps);
  if (!ws) return fail(FLAREPP_ERR_WORKSPACE, "workspace is NULL");
  TRY(check_ptr(ws, "ws"));
  const BlockBwdWs w = block_bwd_ws(ws, dtype, B, N, C, H, M);
  if (ws_bytes < w.bytes)
    return fail(FLAREPP_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, w.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  flarepp::LayerNormParams lp{};
  lp.x = X; lp.gamma = gamma; lp.beta = beta; lp.y = w.xn; lp.T = B * N; lp.C = (int)C; lp.eps = eps;
  lp.mean = w.mean; lp.rstd = w.rstd;
  flarepp::LayerNormBwdParams lb{};
  lb.x = X; lb.gamma = gamma; lb.mean = w.mean; lb.rstd = w.rstd; lb.dxn = w.dxn; lb.dO = dO; lb.dx = dX;
  lb.part = w.part; lb.T = B * N; lb.C = (int)C; lb.nchunks = w.nchunks; lb.chunk = w.chunk;
  float* dgb[2] = {dgamma, dbeta};
  if (dtype == FLAREPP_F32) {
    HIPTRY(flarepp::launch_layernorm<float>(lp, s));
    TRY(backward_impl<float>(dtype, B, N, C, H, M, w.xn, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, w.dxn, dWk, dWv, dWkt,
                             dWvt, dWo, dseeds, nullptr, nullptr, w.ws, w.ws_bytes, s));
    HIPTRY(flarepp::launch_layernorm_bwd<float>(lb, s));
  } else {
    HIPTRY(flarepp::launch_layernorm<__bf16>(lp, s));
    TRY(backward_impl<__bf16>(dtype, B, N, C, H, M, w.xn, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, w.dxn, dWk, dWv, dWkt,
                              dWvt, dWo, dseeds, nullptr, nullptr, w.ws, w.ws_bytes, s));
    HIPTRY(flarepp::launch_layernorm_bwd<__bf16>(lb, s));
  }
  HIPTRY(flarepp::launch_sum_splits(w.part, dgb, C, w.nchunks, 2, s));
  return ok();
}

int flarepp_mixer_forward_shared(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                 const void* X, const void* Wk, const void* Wv, const void* Wo,
                                 const void* seeds, void* O, void* ws, size_t ws_bytes, void* stream) {
  return mixer_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wk, Wv, Wo, seeds, O, nullptr, nullptr, nullptr, ws,
                     ws_bytes, stream, nullptr, 0);
}

size_t flarepp_mixer_backward_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                              int64_t M) {
  if (check_backward_shape(dtype, B, N, C, H, M) != FLAREPP_OK) return 0;
  return bwd_ws(nullptr, dtype, B, N, C, H, M).bytes;
}

int flarepp_mixer_backward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                           const void* X, const void* Wk, const void* Wv, const void* Wkt,
                           const void* Wvt, const void* Wo, const void* seeds, const void* dO,
                           float* dX, float* dWk, float* dWv, float* dWkt, float* dWvt, float* dWo,
                           float* dseeds, void* ws, size_t ws_bytes, void* stream) {
  return backward_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, dX, dWk, dWv, dWkt, dWvt,
                        dWo, dseeds, nullptr, nullptr, ws, ws_bytes, stream);
}

int flarepp_mixer_backward_debug(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                 const void* X, const void* Wk, const void* Wv, const void* Wkt,
                                 const void* Wvt, const void* Wo, const void* seeds, const void* dO,
                                 float* dX, float* dWk, float* dWv, float* dWkt, float* dWvt,
                                 float* dWo, float* dseeds, float* dZ_out, float* dQ_out, void* ws,
                                 size_t ws_bytes, void* stream) {
  return backward_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, dX, dWk, dWv, dWkt, dWvt,
                        dWo, dseeds, dZ_out, dQ_out, ws, ws_bytes, stream);
}

int flarepp_mixer_forward_train(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                const void* X, const void* Wk, const void* Wv, const void* Wkt, const void* Wvt,
                                const void* Wo, const void* seeds, void* O, void* ws, size_t ws_bytes,
                                void* stream) {
  return forward_train_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, O, ws, ws_bytes, stream);
}

int flarepp_mixer_backward_from_saved(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                      const void* X, const void* Wk, const void* Wv, const void* Wkt,
                                      const void* Wvt, const void* Wo, const void* seeds, const void* dO,
                                      float* dX, float* dWk, float* dWv, float* dWkt, float* dWvt, float* dWo,
                                      float* dseeds, void* ws, size_t ws_bytes, void* stream) {
  return backward_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wkt, Wvt, Wo, seeds, dO, dX, dWk, dWv, dWkt, dWvt,
                        dWo, dseeds, nullptr, nullptr, ws, ws_bytes, stream, false, kBwdReverse);
}

int flarepp_mixer_backward_shared(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                  const void* X, const void* Wk, const void* Wv, const void* Wo,
                                  const void* seeds, const void* dO, float* dX, float* dWk, float* dWv,
                                  float* dWo, float* dseeds, void* ws, size_t ws_bytes, void* stream) {
  return backward_entry(dtype, B, N, C, H, M, X, Wk, Wv, Wk, Wv, Wo, seeds, dO, dX, dWk, dWv, nullptr, nullptr,
                        dWo, dseeds, nullptr, nullptr, ws, ws_bytes, stream, true);
}

}  // extern "C"
