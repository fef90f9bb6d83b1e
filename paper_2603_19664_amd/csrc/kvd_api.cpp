// C ABI of libkvd: argument validation (host only, before any HIP call), the
// split policy and workspace sizing, and kernel launches.  See include/kvd.h.
#include "kvd.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "kvd_launch.h"

namespace {

thread_local std::string g_last_error;

kvd_status fail(kvd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

#define KVD_TRY(expr)               \
  do {                              \
    kvd_status _st = (expr);        \
    if (_st != KVD_OK) return _st;  \
  } while (0)

size_t elem_size(const kvd_attn_shape* s) { return s->dtype == KVD_BF16 ? 2 : 4; }

kvd_status check_shape(const kvd_attn_shape* s) {
  if (s == nullptr) return fail(KVD_ERR_NULL, "shape is NULL");
  if (s->dtype != KVD_F32 && s->dtype != KVD_BF16) return fail(KVD_ERR_UNSUPPORTED, "dtype %d is not KVD_F32 or KVD_BF16", s->dtype);
  if (s->d_model <= 0 || s->d_model % kvd::kKT != 0)
    return fail(KVD_ERR_SHAPE, "d_model=%d must be a positive multiple of %d", s->d_model, kvd::kKT);
  if (s->head_dim != 64 && s->head_dim != 128 && s->head_dim != 256)
    return fail(KVD_ERR_UNSUPPORTED, "head_dim=%d is not 64, 128 or 256", s->head_dim);
  if (s->n_kv_heads < 1 || s->n_q_heads < 1) return fail(KVD_ERR_SHAPE, "n_q_heads=%d n_kv_heads=%d must be >= 1", s->n_q_heads, s->n_kv_heads);
  if (s->n_kv_heads > 65535) return fail(KVD_ERR_SHAPE, "n_kv_heads=%d exceeds 65535", s->n_kv_heads);
  if (s->n_q_heads % s->n_kv_heads != 0)
    return fail(KVD_ERR_SHAPE, "n_q_heads=%d is not a multiple of n_kv_heads=%d", s->n_q_heads, s->n_kv_heads);
  if (s->n_q_heads / s->n_kv_heads > kvd::kMaxGroup)
    return fail(KVD_ERR_UNSUPPORTED, "group size %d exceeds %d", s->n_q_heads / s->n_kv_heads, kvd::kMaxGroup);
  if (!std::isfinite(s->rms_eps) || s->rms_eps < 0.0f) return fail(KVD_ERR_SHAPE, "rms_eps must be finite and >= 0");
  if (s->w_layout != KVD_W_ROWMAJOR && s->w_layout != KVD_W_PACKED && s->w_layout != KVD_W_PACKED_GAMMA)
    return fail(KVD_ERR_UNSUPPORTED, "w_layout %d is not a kvd_weight_layout", s->w_layout);
  if (s->w_layout != KVD_W_ROWMAJOR && s->dtype != KVD_BF16)
    return fail(KVD_ERR_UNSUPPORTED, "packed weights are bf16 only");
  if (!std::isfinite(s->rope_theta) || s->rope_theta <= 0.0) return fail(KVD_ERR_SHAPE, "rope_theta must be finite and > 0");
  return KVD_OK;
}

kvd_status check_ptr(const void* p, const char* name) {
  if (p == nullptr) return fail(KVD_ERR_NULL, "%s is NULL", name);
  if ((reinterpret_cast<uintptr_t>(p) & 15u) != 0) return fail(KVD_ERR_ALIGN, "%s is not 16-byte aligned", name);
  return KVD_OK;
}

// gamma is read unless the weights have it folded in (KVD_W_PACKED_GAMMA).
kvd_status check_gamma(const kvd_attn_shape* s, const void* gamma) {
  return s->w_layout == KVD_W_PACKED_GAMMA ? KVD_OK : check_ptr(gamma, "gamma");
}

kvd_status check_view(const kvd_kv_view* v, int32_t T, const char* name) {
  if (v == nullptr) return fail(KVD_ERR_NULL, "%s is NULL", name);
  std::string nk = std::string(name) + "->k", nv = std::string(name) + "->v";
  KVD_TRY(check_ptr(v->k, nk.c_str()));
  KVD_TRY(check_ptr(v->v, nv.c_str()));
  if (v->t_off < 0 || v->t_cap < 1 || (int64_t)v->t_off + T > v->t_cap)
    return fail(KVD_ERR_SHAPE, "%s rows t_off=%d .. t_off+%d exceed t_cap=%d", name, v->t_off, T, v->t_cap);
  return KVD_OK;
}

// A stored tail of T rows read as a ring: rows t_off .. t_off+T-1 modulo t_cap
// (t_off < t_cap, T <= t_cap).  A view with t_off + T <= t_cap is an ordinary
// contiguous block.
kvd_status check_ring_view(const kvd_kv_view* v, int32_t T, const char* name) {
  if (v == nullptr) return fail(KVD_ERR_NULL, "%s is NULL", name);
  std::string nk = std::string(name) + "->k", nv = std::string(name) + "->v";
  KVD_TRY(check_ptr(v->k, nk.c_str()));
  KVD_TRY(check_ptr(v->v, nv.c_str()));
  if (v->t_cap < 1 || v->t_off < 0 || v->t_off >= v->t_cap || T > v->t_cap)
    return fail(KVD_ERR_SHAPE, "%s: %d rows from slot t_off=%d of a ring of t_cap=%d slots (need 0 <= t_off < t_cap "
                "and T <= t_cap)", name, T, v->t_off, v->t_cap);
  return KVD_OK;
}

kvd_status check_batch(int32_t B) {
  if (B < 0 || B > 65535) return fail(KVD_ERR_SHAPE, "B=%d must be in [0, 65535]", B);
  return KVD_OK;
}

void fill_rev(const kvd_attn_shape* s, double* rev) {
  const int pairs = s->head_dim / 2;
  for (int i = 0; i < kvd::kMaxPairs; ++i)
    rev[i] = i < pairs ? std::pow(s->rope_theta, -2.0 * i / s->head_dim) / (2.0 * M_PI) : 0.0;
}

int32_t ceil_div(int64_t a, int64_t b) { return (int32_t)((a + b - 1) / b); }

// Workgroups the bf16 stored-K/V attention's split policy aims for
// (kvd_set_attn_workgroups).
std::atomic<int32_t> g_attn_target{kvd::kSaTargetWgs};

kvd::SaSplit stream_split(const kvd_attn_shape* s, int32_t B, int32_t T) {
  return kvd::sa_split((long long)B * s->n_kv_heads, T, g_attn_target.load(std::memory_order_relaxed));
}

// Token tile of the fused call (kvd_set_fused_tokens): 0 = chosen per call.
std::atomic<int32_t> g_fused_tokens{0};

// The fused call's tiling: the engine (kvd::kFusedTile64 / kFusedWide /
// kFusedSplit), mt recomputed tokens per tile (kMtBf16 / kMtF32, kMtWide or
// kMtSplit), n_rec recomputed tiles, n_tail stored-tail tiles, S = n_rec +
// n_tail splits.
struct FusedPlan {
  int32_t engine, mt, n_rec, n_tail, S;
};

// The wide engine exists for bf16 at head_dim 128 / 256 where its LDS fits.
bool wide_supported(const kvd_attn_shape* s) {
  if (s->dtype != KVD_BF16 || (s->head_dim != 128 && s->head_dim != 256)) return false;
  return kvd::fused_wide_lds_bytes(s->n_q_heads / s->n_kv_heads, s->head_dim) + kvd::gamma_lds_bytes(s->d_model) <=
         kvd::kLdsPerGroup;
}

FusedPlan narrow_plan(const kvd_attn_shape* s, int32_t T_rec, int32_t T_tail) {
  FusedPlan p{};
  p.engine = kvd::kFusedTile64;
  p.mt = kvd::kMtBf16;
  p.n_rec = ceil_div(T_rec, p.mt);
  p.n_tail = s->dtype == KVD_BF16 ? kvd::fused_tail_tiles<uint16_t>(p.n_rec, T_tail)
                                  : kvd::fused_tail_tiles<float>(p.n_rec, T_tail);
  p.S = p.n_rec + p.n_tail;
  return p;
}

FusedPlan wide_plan(int32_t T_rec, int32_t T_tail) {
  FusedPlan p{};
  p.engine = kvd::kFusedWide;
  p.mt = kvd::kMtWide;
  p.n_rec = ceil_div(T_rec, p.mt);
  p.n_tail = kvd::fused_tail_tiles<uint16_t>(p.n_rec, T_tail);
  p.S = p.n_rec + p.n_tail;
  return p;
}

// Two KV heads per 128-token tile: bf16 at head_dim 128 with an even n_kv,
// where the pair tile's LDS fits.  Chunks and splits are the wide engine's.
bool pair_supported(const kvd_attn_shape* s, int32_t T_rec) {
  if (T_rec < 1 || s->dtype != KVD_BF16 || s->head_dim != 128 || s->n_kv_heads % 2 != 0) return false;
  return kvd::fused_pair_lds_bytes(s->n_q_heads / s->n_kv_heads) + kvd::gamma_lds_bytes(s->d_model) <=
         kvd::kLdsPerGroup;
}

FusedPlan pair_plan(int32_t T_rec, int32_t T_tail) {
  FusedPlan p = wide_plan(T_rec, T_tail);
  p.engine = kvd::kFusedPair;
  return p;
}

// The split engine with mt-token chunks: bf16 at head_dim 128 / 256,
// recomputed rows, a tail that folds (at most fold_rows rows), at most
// kSplitMaxChunks chunks per sequence, and its LDS within the limit.
bool split_supported(const kvd_attn_shape* s, int32_t T_rec, int32_t T_tail, int32_t mt) {
  if (s->dtype != KVD_BF16 || (s->head_dim != 128 && s->head_dim != 256)) return false;
  if (T_rec < 1 || T_tail > kvd::fold_rows<uint16_t>() || ceil_div(T_rec, mt) > kvd::kSplitMaxChunks) return false;
  return kvd::fused_split_lds_bytes(s->n_q_heads / s->n_kv_heads, s->head_dim, mt) +
             kvd::gamma_lds_bytes(s->d_model) <= kvd::kLdsPerGroup;
}

FusedPlan split_plan(int32_t T_rec, int32_t mt) {
  FusedPlan p{};
  p.engine = mt == 64 ? kvd::kFusedSplit64 : kvd::kFusedSplit;
  p.mt = mt;
  p.n_rec = ceil_div(T_rec, p.mt);
  p.n_tail = 0;
  p.S = p.n_rec;
  return p;
}

// Wide tiles when supported and the call has at least kWideMinTiles of them (a
// full round of the chip); the split engine with 64-token chunks when 64-token
// tiles of both halves would fill at most kSplit64MaxTiles CUs (twice the
// workgroups, each with half the rows); else 64-token tiles.  With 128-token
// chunks the split engine runs only when asked for: on MI355X, in a 34-layer
// decode step (Gemma-3-4B shape, B = 1, 4096 keys; B = 2, 2048 keys) its
// launches took 58-61 us against 56-57 us on 64-token tiles (its K-loop is no
// faster, and the K-to-V exchange adds a round trip).  kvd_set_fused_tokens
// forces an engine (where it exists).
FusedPlan fused_plan(const kvd_attn_shape* s, int32_t B, int32_t T_rec, int32_t T_tail) {
  const int32_t mode = g_fused_tokens.load(std::memory_order_relaxed);
  const bool wide_ok = T_rec > 0 && wide_supported(s);
  const bool pair_ok = pair_supported(s, T_rec);
  if (mode == kvd::kMtBf16) return narrow_plan(s, T_rec, T_tail);
  if (mode == kvd::kMtWide) return wide_ok ? wide_plan(T_rec, T_tail) : narrow_plan(s, T_rec, T_tail);
  if (mode == KVD_FUSED_PAIR)
    return pair_ok ? pair_plan(T_rec, T_tail) : wide_ok ? wide_plan(T_rec, T_tail) : narrow_plan(s, T_rec, T_tail);
  if (mode == KVD_FUSED_SPLIT)
    return split_supported(s, T_rec, T_tail, kvd::kMtSplit) ? split_plan(T_rec, kvd::kMtSplit)
                                                             : narrow_plan(s, T_rec, T_tail);
  if (mode == KVD_FUSED_SPLIT64)
    return split_supported(s, T_rec, T_tail, 64) ? split_plan(T_rec, 64) : narrow_plan(s, T_rec, T_tail);
  if (pair_ok && (int64_t)B * (s->n_kv_heads / 2) * ceil_div(T_rec, kvd::kMtWide) >= kvd::kWideMinTiles)
    return pair_plan(T_rec, T_tail);
  if (wide_ok && (int64_t)B * s->n_kv_heads * ceil_div(T_rec, kvd::kMtWide) >= kvd::kWideMinTiles)
    return wide_plan(T_rec, T_tail);
  if (split_supported(s, T_rec, T_tail, 64) &&
      (int64_t)B * s->n_kv_heads * ceil_div(T_rec, 64) <= kvd::kSplit64MaxTiles)
    return split_plan(T_rec, 64);
  return narrow_plan(s, T_rec, T_tail);
}

int32_t splits(const kvd_attn_shape* s, int32_t op, int32_t B, int32_t T_main, int32_t T_tail) {
  if (op == KVD_OP_FUSED) return fused_plan(s, B, T_main, T_tail).S;
  return s->dtype == KVD_BF16 ? stream_split(s, B, T_main).S : kvd::decode_splits<float>(T_main);
}

size_t ws_acc_bytes(const kvd_attn_shape* s, int32_t B, int32_t S) {
  return kvd::align_up((size_t)B * s->n_q_heads * S * s->head_dim * sizeof(float), 256);
}
size_t ws_ml_bytes(const kvd_attn_shape* s, int32_t B, int32_t S) {
  return kvd::align_up((size_t)B * s->n_q_heads * S * 2 * sizeof(float), 256);
}
size_t ws_ctr_bytes(const kvd_attn_shape* s, int32_t B) {
  return kvd::align_up((size_t)B * s->n_kv_heads * sizeof(uint64_t), 256);
}
size_t ws_done_bytes(const kvd_attn_shape* s, int32_t B) {
  return ws_ctr_bytes(s, B) + kvd::align_up((size_t)B * s->n_kv_heads * kvd::kSplitBitWords * sizeof(uint64_t), 256);
}
// Workspace: split counters [B][n_kv] uint64 first, then the split engine's
// completion words [B][n_kv][kSplitBitWords] (both zero between calls; their
// place depends on B only, so calls with any key count can share one
// workspace), then partial accumulators [B][n_q][S][hd] fp32 and partial
// (max, sum) [B][n_q][S][2] fp32, then (split engine) the chunks' exchange
// records [B][n_kv][n_rec][xf] fp32.
size_t ws_total(const kvd_attn_shape* s, int32_t B, int32_t S) {
  return ws_done_bytes(s, B) + ws_acc_bytes(s, B, S) + ws_ml_bytes(s, B, S);
}
bool is_split(const FusedPlan& p) { return p.engine == kvd::kFusedSplit || p.engine == kvd::kFusedSplit64; }
size_t ws_xch_bytes(const kvd_attn_shape* s, int32_t B, const FusedPlan& p) {
  return kvd::align_up(
      (size_t)B * s->n_kv_heads * p.n_rec * kvd::split_xf(s->n_q_heads / s->n_kv_heads, p.mt) * sizeof(float), 256);
}
size_t ws_plan_bytes(const kvd_attn_shape* s, int32_t B, const FusedPlan& p) {
  return ws_total(s, B, p.S) + (is_split(p) ? ws_xch_bytes(s, B, p) : 0);
}
float* ws_acc_ptr(const kvd_attn_shape* s, int32_t B, void* ws) {
  return reinterpret_cast<float*>(static_cast<char*>(ws) + ws_done_bytes(s, B));
}
float* ws_ml_ptr(const kvd_attn_shape* s, int32_t B, int32_t S, void* ws) {
  return reinterpret_cast<float*>(static_cast<char*>(ws) + ws_done_bytes(s, B) + ws_acc_bytes(s, B, S));
}
unsigned long long* ws_done_ptr(void* ws) { return static_cast<unsigned long long*>(ws); }

kvd_status check_ws(const kvd_attn_shape* s, int32_t B, int32_t S, void* ws, size_t ws_bytes, size_t extra = 0) {
  const size_t need = ws_total(s, B, S) + extra;
  if (ws == nullptr) return fail(KVD_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return fail(KVD_ERR_ALIGN, "workspace is not 256-byte aligned");
  if (ws_bytes < need) return fail(KVD_ERR_WORKSPACE, "workspace holds %zu bytes, %zu needed", ws_bytes, need);
  return KVD_OK;
}

constexpr size_t kLdsLimit = kvd::kLdsPerGroup;

template <typename T>
size_t attn_lds_need(const kvd_attn_shape* s, bool fused) {
  const int g = s->n_q_heads / s->n_kv_heads;
  const int hd = s->head_dim;
  if (fused) return kvd::fused_lds_bytes<T>(g, hd, sizeof(T) == 2 ? kvd::kMtBf16 : kvd::kMtF32);
  return sizeof(T) == 2 ? kvd::sa_lds(hd, kvd::sa_group(g)).end : kvd::decode_lds_bytes<T>(g, hd);
}

kvd_status check_lds(const kvd_attn_shape* s, bool fused) {
  const size_t need = (s->dtype == KVD_BF16 ? attn_lds_need<uint16_t>(s, fused) : attn_lds_need<float>(s, fused)) +
                      (fused ? kvd::gamma_lds_bytes(s->d_model) : 0);
  if (need > kLdsLimit)
    return fail(KVD_ERR_UNSUPPORTED, "head_dim=%d with group size %d needs %zu bytes of LDS (limit %zu)", s->head_dim,
                s->n_q_heads / s->n_kv_heads, need, kLdsLimit);
  return KVD_OK;
}

kvd_status check_lds_bytes(size_t need, const char* what) {
  if (need > kLdsLimit)
    return fail(KVD_ERR_UNSUPPORTED, "%s needs %zu bytes of LDS for this shape (limit %zu)", what, need, kLdsLimit);
  return KVD_OK;
}

size_t recompute_lds(const kvd_attn_shape* s) {
  const int hd = s->head_dim;
  const size_t base = s->dtype == KVD_BF16
                          ? (hd == 64 ? kvd::proj_lds<uint16_t>(64, kvd::kMtBf16).end
                                      : hd == 128 ? kvd::proj_lds<uint16_t>(128, kvd::kMtBf16).end
                                                  : kvd::proj_lds<uint16_t>(256, kvd::kMtBf16).end)
                          : (hd == 64 ? kvd::proj_lds<float>(64, kvd::kMtF32).end
                                      : hd == 128 ? kvd::proj_lds<float>(128, kvd::kMtF32).end
                                                  : kvd::proj_lds<float>(256, kvd::kMtF32).end);
  // bf16 head_dim 128 / 256 may also run on the split engine
  const size_t split = s->dtype == KVD_BF16 && (hd == 128 || hd == 256) ? kvd::split_lds(hd, kvd::kMtSplit).end : 0;
  return std::max(base, split) + kvd::gamma_lds_bytes(s->d_model);
}

kvd_status device_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return KVD_OK;
  return fail(KVD_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

kvd_status attn_common(const kvd_attn_shape* shape, const void* q, const kvd_kv_view* kv, int32_t B, int32_t T,
                       void* out, void* ws, size_t ws_bytes, void* stream, bool cached) {
  KVD_TRY(check_shape(shape));
  if (cached && shape->dtype != KVD_BF16) return fail(KVD_ERR_UNSUPPORTED, "kvd_cached_attn reads a bf16 cache; dtype must be KVD_BF16");
  KVD_TRY(check_batch(B));
  if (T < 1) return fail(KVD_ERR_SHAPE, "T=%d: attention needs at least one key", T);
  KVD_TRY(check_lds(shape, false));
  if (B == 0) return KVD_OK;
  KVD_TRY(check_ptr(q, "q"));
  if (out != nullptr) KVD_TRY(check_ptr(out, "out"));
  KVD_TRY(check_view(kv, T, "kv"));
  const int32_t S = splits(shape, KVD_OP_DECODE_ATTN, B, T, 0);
  KVD_TRY(check_ws(shape, B, S, ws, ws_bytes));
  kvd::AttnArgs a{};
  if (shape->dtype == KVD_BF16) a.nblk = stream_split(shape, B, T).nblk;
  a.q = q;
  a.k = kv->k;
  a.v = kv->v;
  a.t_cap = kv->t_cap;
  a.t_off = kv->t_off;
  a.out = out;
  a.ws_acc = ws_acc_ptr(shape, B, ws);
  a.ws_ml = ws_ml_ptr(shape, B, S, ws);
  a.ws_done = ws_done_ptr(ws);
  a.B = B;
  a.T = T;
  a.n_q = shape->n_q_heads;
  a.n_kv = shape->n_kv_heads;
  a.S = S;
  return device_status(kvd::launch_decode(a, shape->dtype == KVD_BF16, shape->head_dim, (hipStream_t)stream),
                       cached ? "kvd_cached_attn launch" : "kvd_decode_attn launch");
}

}  // namespace

extern "C" {

int kvd_abi_version(void) { return KVD_ABI_VERSION; }

const char* kvd_status_str(kvd_status st) {
  switch (st) {
    case KVD_OK: return "KVD_OK";
    case KVD_ERR_NULL: return "KVD_ERR_NULL";
    case KVD_ERR_SHAPE: return "KVD_ERR_SHAPE";
    case KVD_ERR_UNSUPPORTED: return "KVD_ERR_UNSUPPORTED";
    case KVD_ERR_WORKSPACE: return "KVD_ERR_WORKSPACE";
    case KVD_ERR_ALIGN: return "KVD_ERR_ALIGN";
    case KVD_ERR_DEVICE: return "KVD_ERR_DEVICE";
  }
  return "KVD_ERR_UNKNOWN";
}

const char* kvd_last_error(void) { return g_last_error.c_str(); }

kvd_status kvd_recompute_kv(const kvd_attn_shape* shape, const void* h, int32_t h_ld, const void* gamma,
                            const void* w_k, const void* w_v, const int32_t* pos0, int32_t B, int32_t T,
                            const kvd_kv_view* out, void* stream) {
  KVD_TRY(check_shape(shape));
  KVD_TRY(check_batch(B));
  if (T < 0) return fail(KVD_ERR_SHAPE, "T=%d must be >= 0", T);
  if (B == 0 || T == 0) return KVD_OK;
  if (h_ld < T) return fail(KVD_ERR_SHAPE, "h_ld=%d is smaller than T=%d", h_ld, T);
  KVD_TRY(check_lds_bytes(recompute_lds(shape), "kvd_recompute_kv"));
  KVD_TRY(check_ptr(h, "h"));
  KVD_TRY(check_gamma(shape, gamma));
  KVD_TRY(check_ptr(w_k, "w_k"));
  KVD_TRY(check_ptr(w_v, "w_v"));
  if (pos0 == nullptr) return fail(KVD_ERR_NULL, "pos0 is NULL");
  KVD_TRY(check_view(out, T, "out"));
  kvd::ProjArgs a{};
  a.h = h;
  a.gamma = gamma;
  a.w_k = w_k;
  a.w_v = w_v;
  a.pos0 = pos0;
  a.k_out = out->k;
  a.v_out = out->v;
  a.h_ld = h_ld;
  a.kv_t_cap = out->t_cap;
  a.kv_t_off = out->t_off;
  a.d = shape->d_model;
  a.n_q = shape->n_q_heads;
  a.n_kv = shape->n_kv_heads;
  a.B = B;
  a.T = T;
  a.n_kv_units = shape->n_kv_heads;
  a.eps = shape->rms_eps;
  fill_rev(shape, a.rev);
  const int G = (long long)B * T <= INT32_MAX ? kvd::stream_group(shape->d_model, B * T, kLdsLimit) : 0;
  const long long stream_wgs =
      G >= 1 ? (long long)(2 * shape->n_kv_heads * shape->head_dim / 32) * (((long long)B * T + G - 1) / G) : 0;
  const long long max_wgs =
      shape->head_dim >= 256 ? kvd::kStreamRecomputeMaxWgsHd256 : kvd::kStreamRecomputeMaxWgs;
  if (shape->dtype == KVD_BF16 && G >= 1 && stream_wgs <= max_wgs)
    return device_status(kvd::launch_project_current(a, 1, shape->head_dim, shape->w_layout, a.n_kv_units,
                                                     (hipStream_t)stream),
                         "kvd_recompute_kv launch");
  return device_status(kvd::launch_proj(a, shape->dtype == KVD_BF16, shape->head_dim, shape->w_layout, a.n_kv_units,
                                        (hipStream_t)stream),
                       "kvd_recompute_kv launch");
}

kvd_status kvd_project_qkv(const kvd_attn_shape* shape, const void* h_new, const void* gamma, const void* w_q,
                           const void* w_k, const void* w_v, const int32_t* pos, int32_t B, void* q_out,
                           const kvd_kv_view* kv_out, void* stream) {
  KVD_TRY(check_shape(shape));
  KVD_TRY(check_batch(B));
  if (shape->dtype == KVD_BF16) {
    // the streaming kernel holds its weight ring and at least one residual row
    if (B > 0 && kvd::stream_group(shape->d_model, B, kLdsLimit) < 1)
      return fail(KVD_ERR_UNSUPPORTED, "kvd_project_qkv needs %zu bytes of LDS for d_model=%d (limit %zu)",
                  kvd::stream_lds(shape->d_model, 1).end, shape->d_model, kLdsLimit);
  } else {
    KVD_TRY(check_lds_bytes(recompute_lds(shape), "kvd_project_qkv"));
  }
  if (B == 0) return KVD_OK;
  KVD_TRY(check_ptr(h_new, "h_new"));
  KVD_TRY(check_gamma(shape, gamma));
  KVD_TRY(check_ptr(w_q, "w_q"));
  KVD_TRY(check_ptr(q_out, "q_out"));
  if (pos == nullptr) return fail(KVD_ERR_NULL, "pos is NULL");
  if (kv_out != nullptr) {
    KVD_TRY(check_ptr(w_k, "w_k"));
    KVD_TRY(check_ptr(w_v, "w_v"));
    KVD_TRY(check_view(kv_out, 1, "kv_out"));
  }
  kvd::ProjArgs a{};
  a.h = h_new;
  a.gamma = gamma;
  a.w_q = w_q;
  a.w_k = w_k;
  a.w_v = w_v;
  a.pos0 = pos;
  a.q_out = q_out;
  if (kv_out) {
    a.k_out = kv_out->k;
    a.v_out = kv_out->v;
    a.kv_t_cap = kv_out->t_cap;
    a.kv_t_off = kv_out->t_off;
  }
  a.h_ld = 1;
  a.d = shape->d_model;
  a.n_q = shape->n_q_heads;
  a.n_kv = shape->n_kv_heads;
  a.B = B;
  a.T = 1;
  a.n_kv_units = kv_out ? shape->n_kv_heads : 0;
  a.eps = shape->rms_eps;
  fill_rev(shape, a.rev);
  const int units = a.n_kv_units + (shape->n_q_heads + 1) / 2;
  return device_status(
      kvd::launch_project_current(a, shape->dtype == KVD_BF16, shape->head_dim, shape->w_layout, units,
                                  (hipStream_t)stream),
      "kvd_project_qkv launch");
}

kvd_status kvd_project_q(const kvd_attn_shape* shape, const void* h_new, const void* gamma, const void* w_q,
                         const int32_t* pos, int32_t B, void* q_out, void* stream) {
  return kvd_project_qkv(shape, h_new, gamma, w_q, nullptr, nullptr, pos, B, q_out, nullptr, stream);
}

kvd_status kvd_decode_attn(const kvd_attn_shape* shape, const void* q, const kvd_kv_view* kv, int32_t B, int32_t T,
                           void* out, void* ws, size_t ws_bytes, void* stream) {
  return attn_common(shape, q, kv, B, T, out, ws, ws_bytes, stream, false);
}

kvd_status kvd_cached_attn(const kvd_attn_shape* shape, const void* q, const kvd_kv_view* kv, int32_t B, int32_t T,
                           void* out, void* ws, size_t ws_bytes, void* stream) {
  return attn_common(shape, q, kv, B, T, out, ws, ws_bytes, stream, true);
}

namespace {

kvd_status check_fused_args(const kvd_attn_shape* shape, const void* q, const void* h, int32_t h_ld,
                            const void* gamma, const void* w_k, const void* w_v, int32_t B, int32_t T_rec,
                            const kvd_kv_view* tail, int32_t T_tail, void* out) {
  KVD_TRY(check_shape(shape));
  KVD_TRY(check_batch(B));
  if (T_rec < 0 || T_tail < 0 || (int64_t)T_rec + T_tail < 1)
    return fail(KVD_ERR_SHAPE, "T_rec=%d T_tail=%d: need T_rec, T_tail >= 0 and at least one key", T_rec, T_tail);
  KVD_TRY(check_lds(shape, true));
  if (B == 0) return KVD_OK;
  KVD_TRY(check_ptr(q, "q"));
  if (out != nullptr) KVD_TRY(check_ptr(out, "out"));
  if (T_rec > 0) {
    if (h_ld < T_rec) return fail(KVD_ERR_SHAPE, "h_ld=%d is smaller than T_rec=%d", h_ld, T_rec);
    KVD_TRY(check_ptr(h, "h"));
    KVD_TRY(check_gamma(shape, gamma));
    KVD_TRY(check_ptr(w_k, "w_k"));
    KVD_TRY(check_ptr(w_v, "w_v"));
  }
  if (T_tail > 0) KVD_TRY(check_ring_view(tail, T_tail, "tail"));
  return KVD_OK;
}

// The fused launch on validated arguments.  pos0 == nullptr: residual row 0 of
// every sequence is at position 0.
kvd_status fused_launch(const kvd_attn_shape* shape, const void* q, const void* h, int32_t h_ld, const void* gamma,
                        const void* w_k, const void* w_v, const int32_t* pos0, int32_t B, int32_t T_rec,
                        const kvd_kv_view* tail, int32_t T_tail, void* out, void* ws, size_t ws_bytes,
                        const kvd_kv_view* kv_debug, void* stream, const char* name) {
  const FusedPlan plan = fused_plan(shape, B, T_rec, T_tail);
  const int32_t S = plan.S;
  // one workgroup per (KV head, sequence, split), indexed in 32 bits
  if ((int64_t)shape->n_kv_heads * B * S > INT32_MAX - 8)
    return fail(KVD_ERR_SHAPE, "%s: n_kv_heads * B * splits = %lld workgroups is too many", name,
                (long long)shape->n_kv_heads * B * S);
  const bool split = is_split(plan);
  KVD_TRY(check_ws(shape, B, S, ws, ws_bytes, split ? ws_xch_bytes(shape, B, plan) : 0));
  kvd::FusedArgs a{};
  a.q = q;
  a.h = h;
  a.h_ld = h_ld;
  a.gamma = gamma;
  a.w_k = w_k;
  a.w_v = w_v;
  a.pos0 = pos0;
  if (T_tail > 0) {
    a.tk = tail->k;
    a.tv = tail->v;
    a.tail_t_cap = tail->t_cap;
    a.tail_t_off = tail->t_off;
  }
  a.T_tail = T_tail;
  if (kv_debug != nullptr && T_rec > 0) {
    a.dbg_k = kv_debug->k;
    a.dbg_v = kv_debug->v;
    a.dbg_t_cap = kv_debug->t_cap;
    a.dbg_t_off = kv_debug->t_off;
  }
  a.ws_acc = ws_acc_ptr(shape, B, ws);
  a.ws_ml = ws_ml_ptr(shape, B, S, ws);
  a.ws_done = ws_done_ptr(ws);
  if (split) {
    a.ws_bits = reinterpret_cast<unsigned long long*>(static_cast<char*>(ws) + ws_ctr_bytes(shape, B));
    a.xch = reinterpret_cast<float*>(static_cast<char*>(ws) + ws_total(shape, B, S));
    a.xf = kvd::split_xf(shape->n_q_heads / shape->n_kv_heads, plan.mt);
  }
  a.out = out;
  a.d = shape->d_model;
  a.n_q = shape->n_q_heads;
  a.n_kv = shape->n_kv_heads;
  a.B = B;
  a.T_rec = T_rec;
  a.n_rec = plan.n_rec;
  a.S = S;
  a.eps = shape->rms_eps;
  fill_rev(shape, a.rev);
  return device_status(kvd::launch_fused(a, shape->dtype == KVD_BF16, shape->head_dim,
                                         shape->w_layout, plan.engine,
                                         (hipStream_t)stream),
                       name);
}

}  // namespace

kvd_status kvd_fused_recompute_attn(const kvd_attn_shape* shape, const void* q, const void* h, int32_t h_ld,
                                    const void* gamma, const void* w_k, const void* w_v, const int32_t* pos0,
                                    int32_t B, int32_t T_rec, const kvd_kv_view* tail, int32_t T_tail, void* out,
                                    void* ws, size_t ws_bytes, const kvd_kv_view* kv_debug, void* stream) {
  KVD_TRY(check_fused_args(shape, q, h, h_ld, gamma, w_k, w_v, B, T_rec, tail, T_tail, out));
  if (B == 0) return KVD_OK;
  if (T_rec > 0) {
    if (pos0 == nullptr) return fail(KVD_ERR_NULL, "pos0 is NULL");
    if (kv_debug != nullptr) KVD_TRY(check_view(kv_debug, T_rec, "kv_debug"));
  }
  return fused_launch(shape, q, h, h_ld, gamma, w_k, w_v, pos0, B, T_rec, tail, T_tail, out, ws, ws_bytes, kv_debug,
                      stream, "kvd_fused_recompute_attn launch");
}

kvd_status kvd_fused_recompute_attn_noalloc(const kvd_attn_shape* shape, const void* q, const void* h, int32_t h_ld,
                                            const void* gamma, const void* w_k, const void* w_v, const int32_t* pos0,
                                            int32_t B, int32_t T_rec, const kvd_kv_view* tail, int32_t T_tail,
                                            void* out, void* stream) {
  KVD_TRY(check_fused_args(shape, q, h, h_ld, gamma, w_k, w_v, B, T_rec, tail, T_tail, out));
  if (B == 0) return KVD_OK;
  if (out == nullptr) return fail(KVD_ERR_NULL, "out is NULL (the no-allocation call always merges its splits)");
  if (T_rec > 0 && pos0 == nullptr) return fail(KVD_ERR_NULL, "pos0 is NULL");
  const size_t need = ws_plan_bytes(shape, B, fused_plan(shape, B, T_rec, T_tail));
  if (need > kvd::kNoAllocScratchBytes)
    return fail(KVD_ERR_WORKSPACE,
                "kvd_fused_recompute_attn_noalloc: B=%d T_rec=%d T_tail=%d needs %zu bytes of scratch, more than the "
                "%zu of the library's static scratch; call kvd_fused_recompute_attn with a workspace instead",
                B, T_rec, T_tail, need, kvd::kNoAllocScratchBytes);
  void* ws = nullptr;
  KVD_TRY(device_status(kvd::noalloc_scratch(&ws), "kvd_fused_recompute_attn_noalloc scratch lookup"));
  // the split counters and completion words start at zero: cleared by a fill
  // kernel (a kernel node under graph capture, never a memset)
  KVD_TRY(device_status(kvd::launch_fill_zero_u64(ws, (int)(ws_done_bytes(shape, B) / sizeof(uint64_t)),
                                                  (hipStream_t)stream),
                        "kvd_fused_recompute_attn_noalloc counter clear"));
  return fused_launch(shape, q, h, h_ld, gamma, w_k, w_v, pos0, B, T_rec, tail, T_tail, out, ws,
                      kvd::kNoAllocScratchBytes, nullptr, stream, "kvd_fused_recompute_attn_noalloc launch");
}

kvd_status kvd_fused_window_attn(const kvd_attn_shape* shape, const void* q, const void* h, int32_t h_ld,
                                 const void* gamma, const void* w_k, const void* w_v, int32_t B, int32_t T_rec,
                                 const kvd_kv_view* tail, int32_t T_tail, int32_t window, void* out, void* ws,
                                 size_t ws_bytes, void* stream) {
  KVD_TRY(check_fused_args(shape, q, h, h_ld, gamma, w_k, w_v, B, T_rec, tail, T_tail, out));
  if (window < 1) return fail(KVD_ERR_SHAPE, "window=%d must be >= 1", window);
  if (B == 0) return KVD_OK;
  // the oldest keys beyond the window go, recomputed rows first; the first kept
  // recomputed row is window index 0
  const int64_t drop = std::max<int64_t>(0, (int64_t)T_rec + T_tail - window);
  const int32_t drop_rec = (int32_t)std::min<int64_t>(drop, T_rec);
  const int32_t drop_tail = (int32_t)(drop - drop_rec);
  const int32_t keep_rec = T_rec - drop_rec, keep_tail = T_tail - drop_tail;
  const size_t elem = shape->dtype == KVD_BF16 ? 2 : 4;
  const void* h_kept = keep_rec > 0 ? static_cast<const char*>(h) + (size_t)drop_rec * shape->d_model * elem : h;
  kvd_kv_view tail_kept{};
  if (keep_tail > 0) {
    tail_kept = *tail;
    tail_kept.t_off = (int32_t)(((int64_t)tail_kept.t_off + drop_tail) % tail_kept.t_cap);
  }
  return fused_launch(shape, q, h_kept, h_ld, gamma, w_k, w_v, nullptr, B, keep_rec,
                      keep_tail > 0 ? &tail_kept : nullptr, keep_tail, out, ws, ws_bytes, nullptr, stream,
                      "kvd_fused_window_attn launch");
}

kvd_status kvd_store_residual(const kvd_attn_shape* shape, const void* h_new, void* ckpt, int32_t c_ld, int32_t row,
                              int32_t B, void* stream) {
  KVD_TRY(check_shape(shape));
  KVD_TRY(check_batch(B));
  if (c_ld < 1 || row < 0 || row >= c_ld)
    return fail(KVD_ERR_SHAPE, "row=%d must lie in the checkpoint store's c_ld=%d rows", row, c_ld);
  if (B == 0) return KVD_OK;
  KVD_TRY(check_ptr(h_new, "h_new"));
  KVD_TRY(check_ptr(ckpt, "ckpt"));
  const size_t row_bytes = (size_t)shape->d_model * elem_size(shape);
  const char* a = static_cast<const char*>(h_new);
  const char* c = static_cast<const char*>(ckpt);
  if (a < c + (size_t)B * c_ld * row_bytes && c < a + (size_t)B * row_bytes)
    return fail(KVD_ERR_SHAPE, "ckpt must not overlap h_new");
  return device_status(kvd::launch_copy_rows(h_new, row_bytes, static_cast<char*>(ckpt) + (size_t)row * row_bytes,
                                             (size_t)c_ld * row_bytes, row_bytes, B, (hipStream_t)stream),
                       "kvd_store_residual launch");
}

kvd_status kvd_pack_matrix(const void* w, int32_t rows, int32_t cols, void* packed, void* stream) {
  if (rows < 32 || rows % 32 != 0) return fail(KVD_ERR_SHAPE, "rows=%d must be a positive multiple of 32", rows);
  if (cols < 16 || cols % 16 != 0) return fail(KVD_ERR_SHAPE, "cols=%d must be a positive multiple of 16", cols);
  KVD_TRY(check_ptr(w, "w"));
  KVD_TRY(check_ptr(packed, "packed"));
  const size_t bytes = (size_t)rows * cols * 2;
  const char* a = static_cast<const char*>(w);
  const char* b = static_cast<const char*>(packed);
  if (a < b + bytes && b < a + bytes) return fail(KVD_ERR_SHAPE, "packed must not overlap w");
  return device_status(kvd::launch_pack(w, nullptr, packed, rows, cols, (hipStream_t)stream), "kvd_pack_matrix launch");
}

namespace {

// Block-forward workspace: q [B][T][n_q][hd], K and V [B][n_kv][T][hd], attention
// heads [B][T][n_q hd], hhat [B][T][d], the MLP activation [B][T][d_ff] (bf16),
// and a vector of ones (the staged operand of the unnormalised projections).
struct BlockWs {
  size_t q, k, v, heads, hhat, u, ones, part, ctr, end;
  kvd::PrefillSplit split;
};
BlockWs block_ws(const kvd_attn_shape* s, int32_t d_ff, int32_t B, int32_t T) {
  const size_t bt = (size_t)B * T, qd = (size_t)s->n_q_heads * s->head_dim;
  BlockWs L{};
  L.q = 0;
  L.k = kvd::align_up(L.q + 2 * bt * qd, 256);
  L.v = kvd::align_up(L.k + 2 * bt * s->n_kv_heads * s->head_dim, 256);
  L.heads = kvd::align_up(L.v + 2 * bt * s->n_kv_heads * s->head_dim, 256);
  L.hhat = kvd::align_up(L.heads + 2 * bt * qd, 256);
  L.u = kvd::align_up(L.hhat + 2 * bt * s->d_model, 256);
  L.ones = kvd::align_up(L.u + 2 * bt * d_ff, 256);
  // the causal attention's key-range parts and their arrival counters (only when it splits)
  L.split = kvd::prefill_split(B, T, s->n_q_heads);
  const size_t blocks = (size_t)B * s->n_q_heads * ((T + 127) / 128);
  const bool split = L.split.NP > 1;
  L.part = kvd::align_up(L.ones + 2 * (size_t)std::max<int64_t>((int64_t)qd, d_ff), 256);
  L.ctr = kvd::align_up(L.part + (split ? 4 * blocks * L.split.NP * kvd::prefill_part_floats(s->head_dim) : 0), 256);
  L.end = kvd::align_up(L.ctr + (split ? 8 * blocks : 0), 256);
  return L;
}

kvd_status check_block(const kvd_attn_shape* shape, int32_t d_ff, int32_t B, int32_t T) {
  KVD_TRY(check_shape(shape));
  KVD_TRY(check_batch(B));
  if (shape->dtype != KVD_BF16) return fail(KVD_ERR_UNSUPPORTED, "the block forward runs in bf16");
  if (shape->w_layout == KVD_W_PACKED_GAMMA)
    return fail(KVD_ERR_UNSUPPORTED, "the block forward takes row-major or packed weights (its norms apply gamma)");
  if (shape->head_dim != 128 && shape->head_dim != 256)
    return fail(KVD_ERR_UNSUPPORTED, "the block forward supports head_dim 128 and 256 (got %d)", shape->head_dim);
  if (shape->d_model % 512 != 0)
    return fail(KVD_ERR_UNSUPPORTED, "the block forward needs d_model %% 512 == 0 (got %d)", shape->d_model);
  if (d_ff < 256 || d_ff % 256 != 0) return fail(KVD_ERR_SHAPE, "d_ff=%d must be a positive multiple of 256", d_ff);
  if ((shape->n_q_heads * shape->head_dim) % kvd::kKT != 0)
    return fail(KVD_ERR_UNSUPPORTED, "n_q_heads * head_dim must be a multiple of %d", kvd::kKT);
  if (T < 0) return fail(KVD_ERR_SHAPE, "T=%d must be >= 0", T);
  if ((int64_t)B * T > INT32_MAX / 2) return fail(KVD_ERR_SHAPE, "B * T = %lld is too large", (long long)B * T);
  const kvd::PrefillSplit sp = kvd::prefill_split(B, T, shape->n_q_heads);
  if ((int64_t)B * shape->n_q_heads * (sp.n_order > 0 ? sp.n_order : (T + 127) / 128) > INT32_MAX)
    return fail(KVD_ERR_SHAPE, "B=%d T=%d n_q_heads=%d: too many attention workgroups", B, T, shape->n_q_heads);
  KVD_TRY(check_lds_bytes(recompute_lds(shape), "kvd_block_forward (projections)"));
  KVD_TRY(check_lds_bytes(kvd::gemm_lds_bytes(std::max(d_ff, shape->n_q_heads * shape->head_dim)),
                          "kvd_block_forward (output projections)"));
  KVD_TRY(check_lds_bytes(kvd::prefill_lds_bytes(shape->head_dim), "kvd_block_forward (attention)"));
  return KVD_OK;
}

}  // namespace

size_t kvd_block_workspace_bytes(const kvd_attn_shape* shape, int32_t d_ff, int32_t B, int32_t T) {
  if (check_block(shape, d_ff, B, T) != KVD_OK) return 0;
  return block_ws(shape, d_ff, B, T).end;
}

kvd_status kvd_block_forward(const kvd_attn_shape* shape, const kvd_block_weights* w, const void* h_in, void* h_out,
                             const int32_t* pos0, int32_t B, int32_t T, void* ws, size_t ws_bytes, void* stream) {
  if (w == nullptr) return fail(KVD_ERR_NULL, "w is NULL");
  KVD_TRY(check_block(shape, w->d_ff, B, T));
  if (B == 0 || T == 0) return KVD_OK;
  KVD_TRY(check_ptr(h_in, "h_in"));
  KVD_TRY(check_ptr(h_out, "h_out"));
  const void* mats[] = {w->gamma_attn, w->w_q, w->w_k, w->w_v, w->w_o, w->gamma_mlp, w->w_gate, w->w_up, w->w_down};
  const char* names[] = {"gamma_attn", "w_q", "w_k", "w_v", "w_o", "gamma_mlp", "w_gate", "w_up", "w_down"};
  for (int i = 0; i < 9; ++i) KVD_TRY(check_ptr(mats[i], names[i]));
  if (pos0 == nullptr) return fail(KVD_ERR_NULL, "pos0 is NULL");
  const size_t hbytes = (size_t)B * T * shape->d_model * 2;
  {
    const char* a = static_cast<const char*>(h_in);
    const char* b = static_cast<const char*>(h_out);
    if (a < b + hbytes && b < a + hbytes) return fail(KVD_ERR_SHAPE, "h_out must not overlap h_in");
  }
  const BlockWs L = block_ws(shape, w->d_ff, B, T);
  if (ws == nullptr) return fail(KVD_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", L.end);
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return fail(KVD_ERR_ALIGN, "workspace is not 256-byte aligned");
  if (ws_bytes < L.end) return fail(KVD_ERR_WORKSPACE, "workspace holds %zu bytes, %zu needed", ws_bytes, L.end);
  char* base = static_cast<char*>(ws);
  const hipStream_t st = (hipStream_t)stream;
  const int packed = shape->w_layout == KVD_W_PACKED;
  const int qd = shape->n_q_heads * shape->head_dim;
  hipError_t e = kvd::launch_fill_ones_bf16(base + L.ones, std::max(qd, w->d_ff), st);
  if (e != hipSuccess) return device_status(e, "kvd_block_forward launch");
  // RMSNorm + Q, K, V of every position (Eqs. q_proj .. v_proj)
  kvd::ProjArgs p{};
  p.h = h_in;
  p.gamma = w->gamma_attn;
  p.w_q = w->w_q;
  p.w_k = w->w_k;
  p.w_v = w->w_v;
  p.pos0 = pos0;
  p.k_out = base + L.k;
  p.v_out = base + L.v;
  p.q_out = base + L.q;
  p.h_ld = T;
  p.kv_t_cap = T;
  p.kv_t_off = 0;
  p.d = shape->d_model;
  p.n_q = shape->n_q_heads;
  p.n_kv = shape->n_kv_heads;
  p.B = B;
  p.T = T;
  p.n_kv_units = shape->n_kv_heads;
  p.eps = shape->rms_eps;
  fill_rev(shape, p.rev);
  e = kvd::launch_proj(p, 1, shape->head_dim, packed, p.n_kv_units + (shape->n_q_heads + 1) / 2, st);
  if (e != hipSuccess) return device_status(e, "kvd_block_forward launch");
  // causal attention (Eqs. attn_weights / head_output)
  kvd::PrefillArgs at{};
  at.q = base + L.q;
  at.k = base + L.k;
  at.v = base + L.v;
  at.out = base + L.heads;
  at.B = B;
  at.T = T;
  at.n_q = shape->n_q_heads;
  at.n_kv = shape->n_kv_heads;
  at.P = L.split.P;
  at.NP = L.split.NP;
  at.n_order = L.split.n_order;
  std::copy(L.split.order, L.split.order + L.split.n_order, at.order);
  if (L.split.NP > 1) {
    at.part = reinterpret_cast<float*>(base + L.part);
    at.ctr = reinterpret_cast<unsigned long long*>(base + L.ctr);
    e = kvd::launch_fill_zero_u64(at.ctr, B * shape->n_q_heads * ((T + 127) / 128), st);
    if (e != hipSuccess) return device_status(e, "kvd_block_forward launch");
  }
  e = kvd::launch_prefill_attn(at, shape->head_dim, st);
  if (e != hipSuccess) return device_status(e, "kvd_block_forward launch");
  // hhat = h + heads W_o (Eq. attn_sublayer)
  kvd::GemmArgs g{};
  g.x = base + L.heads;
  g.gamma = base + L.ones;
  g.w = w->w_o;
  g.res = h_in;
  g.out = base + L.hhat;
  g.M = B * T;
  g.K = qd;
  g.N = shape->d_model;
  g.norm = 0;
  g.eps = shape->rms_eps;
  e = kvd::launch_gemm(g, kvd::kEpiResidual, packed, st);
  if (e != hipSuccess) return device_status(e, "kvd_block_forward launch");
  // u = SiLU(xbar W_gate) * (xbar W_up), xbar = RMSNorm(hhat; gamma_mlp)
  g = kvd::GemmArgs{};
  g.x = base + L.hhat;
  g.gamma = w->gamma_mlp;
  g.w = w->w_gate;
  g.w2 = w->w_up;
  g.out = base + L.u;
  g.M = B * T;
  g.K = shape->d_model;
  g.N = w->d_ff;
  g.norm = 1;
  g.eps = shape->rms_eps;
  e = kvd::launch_gemm(g, kvd::kEpiSwiglu, packed, st);
  if (e != hipSuccess) return device_status(e, "kvd_block_forward launch");
  // h_out = hhat + u W_down (Eq. mlp_sublayer)
  g = kvd::GemmArgs{};
  g.x = base + L.u;
  g.gamma = base + L.ones;
  g.w = w->w_down;
  g.res = base + L.hhat;
  g.out = h_out;
  g.M = B * T;
  g.K = w->d_ff;
  g.N = shape->d_model;
  g.norm = 0;
  g.eps = shape->rms_eps;
  return device_status(kvd::launch_gemm(g, kvd::kEpiResidual, packed, st), "kvd_block_forward launch");
}

kvd_status kvd_pack_weights(const kvd_attn_shape* shape, const void* w, int32_t rows, void* packed, void* stream) {
  if (shape == nullptr) return fail(KVD_ERR_NULL, "shape is NULL");
  kvd_attn_shape s = *shape;
  s.w_layout = KVD_W_ROWMAJOR;
  KVD_TRY(check_shape(&s));
  if (s.dtype != KVD_BF16) return fail(KVD_ERR_UNSUPPORTED, "kvd_pack_weights packs bf16 weights");
  if (rows < 32 || rows % 32 != 0) return fail(KVD_ERR_SHAPE, "rows=%d must be a positive multiple of 32", rows);
  KVD_TRY(check_ptr(w, "w"));
  KVD_TRY(check_ptr(packed, "packed"));
  const size_t bytes = (size_t)rows * s.d_model * 2;
  const char* a = static_cast<const char*>(w);
  const char* b = static_cast<const char*>(packed);
  if (a < b + bytes && b < a + bytes) return fail(KVD_ERR_SHAPE, "packed must not overlap w");
  return device_status(kvd::launch_pack(w, nullptr, packed, rows, s.d_model, (hipStream_t)stream), "kvd_pack_weights launch");
}

kvd_status kvd_pack_weights_gamma(const kvd_attn_shape* shape, const void* w, const void* gamma, int32_t rows,
                                  void* packed, void* stream) {
  if (shape == nullptr) return fail(KVD_ERR_NULL, "shape is NULL");
  kvd_attn_shape s = *shape;
  s.w_layout = KVD_W_ROWMAJOR;
  KVD_TRY(check_shape(&s));
  if (s.dtype != KVD_BF16) return fail(KVD_ERR_UNSUPPORTED, "kvd_pack_weights_gamma packs bf16 weights");
  if (rows < 32 || rows % 32 != 0) return fail(KVD_ERR_SHAPE, "rows=%d must be a positive multiple of 32", rows);
  KVD_TRY(check_ptr(w, "w"));
  KVD_TRY(check_ptr(gamma, "gamma"));
  KVD_TRY(check_ptr(packed, "packed"));
  const size_t bytes = (size_t)rows * s.d_model * 2;
  const char* a = static_cast<const char*>(w);
  const char* b = static_cast<const char*>(packed);
  const char* g = static_cast<const char*>(gamma);
  if (a < b + bytes && b < a + bytes) return fail(KVD_ERR_SHAPE, "packed must not overlap w");
  if (g < b + bytes && b < g + (size_t)s.d_model * 2) return fail(KVD_ERR_SHAPE, "packed must not overlap gamma");
  return device_status(kvd::launch_pack(w, gamma, packed, rows, s.d_model, (hipStream_t)stream),
                       "kvd_pack_weights_gamma launch");
}

kvd_status kvd_combine(const kvd_attn_shape* shape, int32_t B, int32_t S, const void* ws, size_t ws_bytes, void* out,
                       void* stream) {
  KVD_TRY(check_shape(shape));
  KVD_TRY(check_batch(B));
  if (S < 1) return fail(KVD_ERR_SHAPE, "S=%d must be >= 1", S);
  if (B == 0) return KVD_OK;
  KVD_TRY(check_ptr(out, "out"));
  KVD_TRY(check_ws(shape, B, S, const_cast<void*>(ws), ws_bytes));
  const float* acc = ws_acc_ptr(shape, B, const_cast<void*>(ws));
  const float* ml = ws_ml_ptr(shape, B, S, const_cast<void*>(ws));
  return device_status(kvd::launch_combine(acc, ml, out, shape->n_q_heads, B, S, shape->dtype == KVD_BF16,
                                           shape->head_dim, (hipStream_t)stream),
                       "kvd_combine launch");
}

int32_t kvd_num_splits(const kvd_attn_shape* shape, int32_t op, int32_t B, int32_t T_main, int32_t T_tail) {
  if (check_shape(shape) != KVD_OK || B < 0 || T_main < 0 || T_tail < 0) return 0;
  if (op == KVD_OP_FUSED) {
    if ((int64_t)T_main + T_tail < 1) return 0;
  } else if (op == KVD_OP_DECODE_ATTN || op == KVD_OP_CACHED_ATTN) {
    if (T_main < 1 || T_tail != 0) return 0;
  } else {
    return 0;
  }
  return splits(shape, op, B, T_main, T_tail);
}

int32_t kvd_set_attn_workgroups(int32_t target) {
  if (target <= 0) target = kvd::kSaTargetWgs;
  target = std::min<int32_t>(target, 1 << 22);
  return g_attn_target.exchange(target, std::memory_order_relaxed);
}

int32_t kvd_set_fused_tokens(int32_t tokens) {
  if (tokens != kvd::kMtBf16 && tokens != kvd::kMtWide && tokens != KVD_FUSED_SPLIT && tokens != KVD_FUSED_SPLIT64 &&
      tokens != KVD_FUSED_PAIR)
    tokens = 0;
  return g_fused_tokens.exchange(tokens, std::memory_order_relaxed);
}

size_t kvd_workspace_bytes(const kvd_attn_shape* shape, int32_t op, int32_t B, int32_t T_main, int32_t T_tail) {
  int32_t S = kvd_num_splits(shape, op, B, T_main, T_tail);
  if (S == 0) return 0;
  // fused: enough for either tiling, so that the size grows with T_rec and
  // T_tail whichever tile each call gets
  if (op == KVD_OP_FUSED) {
    size_t n = ws_plan_bytes(shape, B, narrow_plan(shape, T_main, T_tail));
    if (T_main > 0 && wide_supported(shape)) n = std::max(n, ws_plan_bytes(shape, B, wide_plan(T_main, T_tail)));
    if (split_supported(shape, T_main, T_tail, kvd::kMtSplit))
      n = std::max(n, ws_plan_bytes(shape, B, split_plan(T_main, kvd::kMtSplit)));
    if (split_supported(shape, T_main, T_tail, 64)) n = std::max(n, ws_plan_bytes(shape, B, split_plan(T_main, 64)));
    return n;
  }
  return ws_total(shape, B, S);
}

}  // extern "C"
