// Kernels and launchers of libkvd (gfx950).
//
//   proj_kernel         RMSNorm + projection + RoPE of token tiles (RECOMPUTE_KV /
//                       prefill; also the fp32 current-token projection).
//   stream_proj_kernel  bf16 current-token q, K_t, V_t of a decode step (a GEMV
//                       shape): four waves per 32 weight rows stream them into an
//                       LDS ring, one runs the MFMA chain; the same per-element
//                       arithmetic as proj_kernel.
//   fused_kernel        per (b, KV head, 64-key chunk): recompute K/V of the chunk
//                       into LDS and emit its split-K softmax partial without writing
//                       K/V to HBM; stored tail tiles (CONCAT) ride along.
//   fused_wide_kernel   the same per 128-key chunk (bf16, head_dim 128 / 256).
//   fused_pair_kernel   the same per (b, pair of KV heads, 128-key chunk) at bf16
//                       head_dim 128, on the head_dim 256 wave layout.
//   fused_split_kernel  the same with a chunk's K and V rows recomputed by two
//                       workgroups (one half each).
//   proj_split_kernel / proj_wide_kernel  prefill on the split / wide layouts.
//   stream_attn_kernel  bf16 stored-K/V attention: per (key split, KV head, b) one
//                       workgroup streams the split's keys in 16-key blocks, loads of
//                       the next block in flight, and emits one split-K partial.
//   decode_kernel       fp32 stored-K/V attention, per (b, KV head, 64-key chunk).
//   combine_kernel      merges the partials of each (b, query head) in split order.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "kvd_device.hpp"
#include "kvd_launch.h"

namespace kvd {

// ------------------------------------------------------------------ recompute / prefill

// grid: xcd_map(n_units * n_tiles) workgroups; item = unit * n_tiles + tile, so
// the token tiles of one KV head (which share W_k / W_v) run on one XCD.
template <typename T, int HD, int MT, bool PACKED, bool FOLD>
__global__ __launch_bounds__(kNtTile, 1) void proj_kernel(ProjArgs a, int per_xcd, int n_tiles, int n_units) {
  extern __shared__ __align__(16) char lds[];
  constexpr int NT = kNtTile;
  constexpr ProjLds PL = proj_lds<T>(HD, MT);
  constexpr int CPT = MT * 8 / NT;
  constexpr int KLD = kv_ld<T>(HD);
  const int tid = threadIdx.x;
  // 32-bit index arithmetic: the launch's grid bounds the item count
  const unsigned item = (blockIdx.x % kXcds) * (unsigned)per_xcd + blockIdx.x / kXcds;
  if (item >= (unsigned)n_units * (unsigned)n_tiles) return;
  const int unit = (int)(item / (unsigned)n_tiles);
  const int tile = (int)(item - (unsigned)unit * (unsigned)n_tiles);

  double* rev = reinterpret_cast<double*>(lds + PL.rev);
  float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
  int* pos = reinterpret_cast<int*>(lds + PL.pos);
  T* hst = reinterpret_cast<T*>(lds + PL.hst);
  T* kv = reinterpret_cast<T*>(lds + PL.kv);

  const long long ntok = (long long)a.B * a.T;
  const long long n0 = (long long)tile * MT;
  const bool kv_mode = unit < a.n_kv_units;
  const size_t hd_d = (size_t)HD * a.d;

  Half halves[2];
  int heads[2];
  if (kv_mode) {
    halves[0] = Half{static_cast<const T*>(a.w_k) + unit * hd_d, 1};
    halves[1] = Half{static_cast<const T*>(a.w_v) + unit * hd_d, 0};
    heads[0] = heads[1] = unit;
  } else {
    const int u = unit - a.n_kv_units;
    heads[0] = 2 * u;
    heads[1] = 2 * u + 1;
    halves[0] = Half{static_cast<const T*>(a.w_q) + heads[0] * hd_d, 1};
    halves[1] = Half{heads[1] < a.n_q ? static_cast<const T*>(a.w_q) + heads[1] * hd_d : nullptr, 1};
  }

  // gamma, rev and the positions reach LDS while the K-loop's first loads are in flight
  uint16_t* gam = reinterpret_cast<uint16_t*>(lds + PL.end);
  const TileSetup<T, HD, NT, false, !FOLD> su(nullptr, 0, 0, 0, 0, a.gamma, a.d, a.rev);
  // position of staged token tid (tid < MT): pos0[b] + t, 0 past the end; the
  // load is issued here and its value used in setup()
  const long long pn = n0 + min(tid, MT - 1);
  const bool pok = pn < ntok;
  const int pb = pok ? (int)(pn / a.T) : 0;
  const int pt = pok ? (int)(pn - (long long)pb * a.T) : 0;
  const int pbase = a.pos0[pb];
  auto setup = [&]() {
    su.store(nullptr, gam, rev);
    if (tid < MT) pos[tid] = pok ? pbase + pt : 0;
  };
  const T* hrow[CPT];
  bool valid[CPT];
#pragma unroll
  for (int r = 0; r < CPT; ++r) {
    long long n = n0 + (tid >> 3) + (NT / 8) * r;
    valid[r] = n < ntok;
    if (!valid[r]) n = n0;  // any readable row; its values are replaced by zeros
    const int b = (int)(n / a.T), t = (int)(n - (long long)b * a.T);
    hrow[r] = static_cast<const T*>(a.h) + ((size_t)b * a.h_ld + t) * a.d + 8 * (tid & 7);
  }

  if constexpr (sizeof(T) == 2) {
    MfmaTile<HD, MT, PACKED, FOLD>::run(hrow, valid, gam, static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves,
                                        hst, rinv, pos, rev, kv, setup);
  } else {
    F32Tile<HD, MT>::run(hrow, valid, static_cast<const float*>(a.gamma), a.d, a.eps, halves, hst, rinv, pos, rev,
                         kv, setup);
  }
  __syncthreads();

  // store: 16-byte chunks of each valid token row of each present half.
  constexpr int CH = 16 / sizeof(T);
  constexpr int CPR = HD / CH;
  for (int c = tid; c < 2 * MT * CPR; c += NT) {
    const int half = c / (MT * CPR);
    const int rem = c - half * MT * CPR;
    const int row = rem / CPR, ch = rem - row * CPR;
    const long long n = n0 + row;
    const bool present = half ? halves[1].w != nullptr : halves[0].w != nullptr;
    if (n >= ntok || !present) continue;
    const int b = (int)(n / a.T), t = (int)(n - (long long)b * a.T);
    const int head = half ? heads[1] : heads[0];
    T* dst;
    if (kv_mode) {
      T* base = static_cast<T*>(half ? a.v_out : a.k_out);
      dst = base + (((size_t)b * a.n_kv + head) * a.kv_t_cap + a.kv_t_off + t) * HD;
    } else {
      dst = static_cast<T*>(a.q_out) + (((size_t)b * a.T + t) * a.n_q + head) * HD;  // [B][T][n_q][hd]
    }
    *reinterpret_cast<uint4*>(dst + ch * CH) =
        *reinterpret_cast<const uint4*>(kv + (size_t)row * KLD + half * HD + ch * CH);
  }
}

// ------------------------------------------------------------------ recompute / prefill, wide tiles

// bf16, head_dim 128 / 256, for calls with at least a full round of 128-token
// tiles: WideTile's 128-token tile of both halves of a unit (a KV head's K and
// V rows, or query heads 2u and 2u + 1) for up to 128 tokens of one sequence.
// grid: xcd_map(n_units * B * tps) with tps = ceil(T / 128); item = (unit * B +
// b) * tps + tile, so a unit's tiles run on one XCD.  Per element the
// arithmetic is the other engines' (the same MFMA chain over d, staging, 1/rms
// and epilogue), so the K/V are bit-identical.
template <int HD, bool PACKED, bool FOLD>
__global__ __launch_bounds__(kNtWide, 1) void proj_wide_kernel(ProjArgs a, int per_xcd, int tps, int n_units) {
  extern __shared__ __align__(16) char lds[];
  constexpr int MT = kMtWide, NT = kNtWide;
  constexpr ProjLds PL = proj_lds<uint16_t>(HD, MT);
  constexpr int KLD = kv_ld<uint16_t>(HD);
  const int tid = threadIdx.x;
  const unsigned item = (blockIdx.x % kXcds) * (unsigned)per_xcd + blockIdx.x / kXcds;
  const unsigned n_tiles = (unsigned)a.B * (unsigned)tps;
  if (item >= (unsigned)n_units * n_tiles) return;
  const int unit = (int)(item / n_tiles);
  const unsigned rem = item - (unsigned)unit * n_tiles;
  const int b = (int)(rem / (unsigned)tps);
  const int t0 = (int)(rem - (unsigned)b * (unsigned)tps) * MT;
  const int n = min(MT, a.T - t0);
  const size_t hd_d = (size_t)HD * a.d;
  const bool kv_mode = unit < a.n_kv_units;
  Half halves[2];
  int heads[2];
  if (kv_mode) {
    halves[0] = Half{static_cast<const uint16_t*>(a.w_k) + unit * hd_d, 1};
    halves[1] = Half{static_cast<const uint16_t*>(a.w_v) + unit * hd_d, 0};
    heads[0] = heads[1] = unit;
  } else {
    const int u = unit - a.n_kv_units;
    heads[0] = 2 * u;
    heads[1] = 2 * u + 1;
    halves[0] = Half{static_cast<const uint16_t*>(a.w_q) + heads[0] * hd_d, 1};
    halves[1] = Half{heads[1] < a.n_q ? static_cast<const uint16_t*>(a.w_q) + heads[1] * hd_d : nullptr, 1};
  }

  double* rev = reinterpret_cast<double*>(lds + PL.rev);
  float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
  int* pos = reinterpret_cast<int*>(lds + PL.pos);
  uint16_t* hst = reinterpret_cast<uint16_t*>(lds + PL.hst);
  uint16_t* kv = reinterpret_cast<uint16_t*>(lds + PL.kv);
  uint16_t* gam = reinterpret_cast<uint16_t*>(lds + PL.end);
  const TileSetup<uint16_t, HD, NT, false, !FOLD> su(nullptr, 0, 0, 0, 0, a.gamma, a.d, a.rev);
  auto setup = [&]() {
    su.store(nullptr, gam, rev);
    if (tid < MT) pos[tid] = a.pos0[b] + t0 + tid;
  };
  WideTile<HD, MT, PACKED, FOLD, kNtWide, kv_ld<uint16_t>(HD), false, true>::run(
      static_cast<const uint16_t*>(a.h) + ((size_t)b * a.h_ld + t0) * a.d, n, gam,
      static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves, hst, rinv, pos, rev, kv, setup);
  __syncthreads();

  // store: 16-byte chunks of each valid token row of each present half
  constexpr int CPR = HD / 8;
  for (int c = tid; c < 2 * n * CPR; c += NT) {
    const int half = c / (n * CPR);
    const int r2 = c - half * n * CPR;
    const int row = r2 / CPR, ch = r2 - row * CPR;
    if (half ? halves[1].w == nullptr : halves[0].w == nullptr) continue;
    const int head = heads[half];
    uint16_t* dst;
    if (kv_mode) {
      uint16_t* base = static_cast<uint16_t*>(half ? a.v_out : a.k_out);
      dst = base + (((size_t)b * a.n_kv + head) * a.kv_t_cap + a.kv_t_off + t0 + row) * HD;
    } else {
      dst = static_cast<uint16_t*>(a.q_out) + (((size_t)b * a.T + t0 + row) * a.n_q + head) * HD;  // [B][T][n_q][hd]
    }
    *reinterpret_cast<uint4*>(dst + ch * 8) = *reinterpret_cast<const uint4*>(kv + (size_t)row * KLD + half * HD + ch * 8);
  }
}

// ------------------------------------------------------------------ recompute / prefill, split engine

// bf16, head_dim 128 / 256: RW rows of one half of a unit (a KV head's K rows
// or its V rows; query heads 2u and 2u + 1 for a q unit) for a tile of up to MT
// tokens of one sequence, per workgroup of NT threads: RW = HD (the split
// engine, MT = kMtSplit) or, for calls too small to fill the chip, RW = 128 and
// MT = 64 (the narrow tile: more, shorter workgroups).  grid: xcd_map(2 * RG *
// n_units * B * tps) with RG = HD / RW row groups and tps = ceil(T / MT) tiles
// per sequence; item = (((unit * B + b) * tps + tile) * 2 + half) * RG + rg, so
// the row groups and the two halves of a tile are adjacent items on one XCD
// (its L2 serves the tile's residual rows to all of them) and a unit's tiles
// stay on one XCD.  Per element the arithmetic is the other engines' (the same
// MFMA chain over d, staging, 1/rms and epilogue), so the K/V are
// bit-identical.
template <int HD, int MT, int NT, int RW, bool PACKED, bool FOLD>
__global__ __launch_bounds__(NT, 1) void proj_split_kernel(ProjArgs a, int per_xcd, int tps, int n_units) {
  extern __shared__ __align__(16) char lds[];
  constexpr int RG = HD / RW;
  constexpr ProjLds PL = split_lds(RW, MT);
  constexpr int KLD = split_ld(RW);
  static_assert(RG * RW == HD, "row groups");
  const int tid = threadIdx.x;
  const unsigned item = (blockIdx.x % kXcds) * (unsigned)per_xcd + blockIdx.x / kXcds;
  const unsigned n_tiles = (unsigned)a.B * (unsigned)tps;
  if (item >= 2u * RG * (unsigned)n_units * n_tiles) return;
  const int rg = (int)(item % RG);
  const unsigned ih = item / RG;
  const int half = (int)(ih & 1u);
  const unsigned ut = ih >> 1;
  const int unit = (int)(ut / n_tiles);
  const unsigned rem = ut - (unsigned)unit * n_tiles;
  const int b = (int)(rem / (unsigned)tps);
  const int t0 = (int)(rem - (unsigned)b * (unsigned)tps) * MT;
  const int n = min(MT, a.T - t0);
  const size_t hd_d = (size_t)HD * a.d;
  const bool kv_mode = unit < a.n_kv_units;
  const int head = kv_mode ? unit : 2 * (unit - a.n_kv_units) + half;
  if (!kv_mode && head >= a.n_q) return;
  const uint16_t* w = (kv_mode ? static_cast<const uint16_t*>(half ? a.w_v : a.w_k) + head * hd_d
                               : static_cast<const uint16_t*>(a.w_q) + head * hd_d) +
                      (size_t)rg * RW * a.d;
  const Half halves[2] = {Half{w, kv_mode ? 1 - half : 1}, Half{nullptr, 0}};

  double* rev = reinterpret_cast<double*>(lds + PL.rev);
  float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
  int* pos = reinterpret_cast<int*>(lds + PL.pos);
  uint16_t* hst = reinterpret_cast<uint16_t*>(lds + PL.hst);
  uint16_t* kv = reinterpret_cast<uint16_t*>(lds + PL.kv);
  uint16_t* gam = reinterpret_cast<uint16_t*>(lds + PL.end);
  const TileSetup<uint16_t, HD, NT, false, !FOLD> su(nullptr, 0, 0, 0, 0, a.gamma, a.d, a.rev);
  auto setup = [&]() {
    su.store(nullptr, gam, rev);
    if (tid < MT) pos[tid] = a.pos0[b] + t0 + tid;
  };
  // the row group's RoPE frequencies start at pair rg * RW / 2
  WideTile<RW, MT, PACKED, FOLD, NT, KLD, true>::run(static_cast<const uint16_t*>(a.h) + ((size_t)b * a.h_ld + t0) * a.d, n,
                                               gam, static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves, hst,
                                               rinv, pos, rev + rg * (RW / 2), kv, setup);
  __syncthreads();

  // store: 16-byte chunks of the tile's valid rows (columns rg * RW ..)
  constexpr int CPR = RW / 8;
  uint16_t* dst0;
  size_t row_stride;
  if (kv_mode) {
    dst0 = static_cast<uint16_t*>(half ? a.v_out : a.k_out) +
           (((size_t)b * a.n_kv + head) * a.kv_t_cap + a.kv_t_off + t0) * HD + rg * RW;
    row_stride = HD;
  } else {
    dst0 = static_cast<uint16_t*>(a.q_out) + (((size_t)b * a.T + t0) * a.n_q + head) * HD + rg * RW;  // [B][T][n_q][hd]
    row_stride = (size_t)a.n_q * HD;
  }
  for (int c = tid; c < n * CPR; c += NT) {
    const int row = c / CPR, ch = c - row * CPR;
    *reinterpret_cast<uint4*>(dst0 + row * row_stride + ch * 8) =
        *reinterpret_cast<const uint4*>(kv + (size_t)row * KLD + ch * 8);
  }
}

// ------------------------------------------------------------------ streaming current-token projection

// One workgroup of kStreamWaves waves per 32 weight rows.  blockIdx.x: a 32-row
// block of [W_q rows | W_k rows | W_v rows] (no W_q rows without q_out);
// blockIdx.y: a group of G of the B * T tokens (T = 1 for a decode step's
// current tokens; the few rows of a short recompute otherwise).
// Waves 1.. (the loaders) each keep their share of kStreamDepth chunks of the
// rows' MFMA A fragments (1 KiB each) in flight in registers; wave 0 runs the
// MFMA chain over d and issues no global loads in its loop.  Barrier c: the
// loaders have written chunk c + 1 into the LDS ring (slot (c + 1) % NR, whose
// previous chunk wave 0 read before barrier c - 2); after it wave 0 reads chunk
// c + 1 while chunk c's MFMAs run.  The loaders also carry the tokens' sums of
// squares along, chunk by chunk, and write 1/rms before the last barrier: only
// the epilogue needs it.  Per output element the arithmetic is MfmaTile's (the
// same MFMA chain over d, the same sum-of-squares chain, 1/rms and epilogue), so
// K_t / V_t equal what recompute gives for the same row.  NCH > 0: the chunk
// count, fixed at compile time so that the loaders' loop is straight-line code
// (their memory-counter waits then keep every chunk in flight).
template <int HD, bool PACKED, int NCH, bool FOLD>
__global__ __launch_bounds__(64 * kStreamWaves) void stream_proj_kernel(ProjArgs a, int q_blocks, int k_blocks,
                                                                        int G) {
  extern __shared__ __align__(16) char lds[];
  constexpr int NW = kStreamWaves, CK = kStreamChunk, NR = kStreamSlots, D = kStreamDepth;
  constexpr int FPC = 4 * CK;          // A fragments per chunk
  constexpr int LPW = FPC / (NW - 1);  // fragments per loader wave per chunk
  static_assert(FPC % (NW - 1) == 0 && NR >= 3, "ring");
  static_assert(8 * (NW - 1) >= kProjTok, "a sum-of-squares row per 8 loader lanes");
  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int d = a.d;
  const StreamLds SL = stream_lds(d, G);
  const int HLD = stream_h_ld(d);
  double* rev = reinterpret_cast<double*>(lds + SL.rev);
  float* rinv = reinterpret_cast<float*>(lds + SL.rinv);
  int* pos = reinterpret_cast<int*>(lds + SL.pos);
  uint16_t* gl = reinterpret_cast<uint16_t*>(lds + SL.gam);
  uint16_t* ring = reinterpret_cast<uint16_t*>(lds + SL.ring);
  uint16_t* hb = reinterpret_cast<uint16_t*>(lds + SL.hb);
  uint16_t* hs = reinterpret_cast<uint16_t*>(lds + SL.hs);

  const int blk = blockIdx.x;
  // tokens n0 .. n0 + nt - 1 of the B * T: token n is row t = n % T of sequence b = n / T
  const int n0 = blockIdx.y * G;
  const int nt = min(G, a.B * a.T - n0);
  const uint16_t* W;
  int row0, rope, mat;  // mat: 0 q, 1 k, 2 v
  if (blk < q_blocks) {
    W = static_cast<const uint16_t*>(a.w_q); row0 = 32 * blk; rope = 1; mat = 0;
  } else if (blk < q_blocks + k_blocks) {
    W = static_cast<const uint16_t*>(a.w_k); row0 = 32 * (blk - q_blocks); rope = 1; mat = 1;
  } else {
    W = static_cast<const uint16_t*>(a.w_v); row0 = 32 * (blk - q_blocks - k_blocks); rope = 0; mat = 2;
  }
  // lane l's 16 bytes of A fragment (K-step s, substep k): row l % 32, columns
  // 16 k + 8 (l / 32) of the K-step (packed: the fragment's contiguous 1 KiB)
  const uint16_t* wrow = PACKED ? W + (size_t)row0 * d + 8 * lane : W + (size_t)(row0 + (lane & 31)) * d + 8 * (lane >> 5);
  const int nsteps = d / kKT;
  const int nchunks = NCH > 0 ? NCH : (nsteps + CK - 1) / CK;
  const int ld = w - 1;  // loader index (waves 1..)
  u32x4_t wr[D][LPW];    // loaders: chunks in flight, chunk c in wr[c % D]
  auto load_chunk = [&](u32x4_t (&rv)[LPW], int c) {
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      const int f = min(c * FPC + ld * LPW + i, 4 * nsteps - 1);
      rv[i] = *reinterpret_cast<const u32x4_t*>(wrow + w_off<PACKED>(f >> 2, f & 3));
    }
  };
  auto store_chunk = [&](const u32x4_t (&rv)[LPW], int c) {
    uint16_t* slot = ring + (size_t)(c % NR) * FPC * 512 + 8 * lane;
#pragma unroll
    for (int i = 0; i < LPW; ++i)
      *reinterpret_cast<u32x4_t*>(slot + (ld * LPW + i) * 512) = rv[i];
  };
  // gamma * h -> bf16 into hs (present rows only), by all waves between barriers A and C
  // (folded weights: the MFMA reads the residual rows in hb as they are)
  auto scale_rows = [&]() {
    if constexpr (FOLD) return;
    const int cpr = d / 8;
    for (int i = tid; i < nt * cpr; i += 64 * NW) {
      const int r = i / cpr, ch = i - r * cpr;
      *reinterpret_cast<uint4*>(hs + (size_t)r * HLD + 8 * ch) =
          scale_chunk_bf16(*reinterpret_cast<const uint4*>(hb + (size_t)r * HLD + 8 * ch),
                           *reinterpret_cast<const uint4*>(gl + 8 * ch));
    }
  };
  f32x16_t acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0f;

  // The two roles run separate code paths with the same sequence of barriers, so
  // that the loaders' memory-counter waits are exact.
  if (w > 0) {
    // The residual rows of the group and gamma straight into LDS (global-to-LDS,
    // one instruction per 1 KiB of a row, rows spread over the loaders), then the
    // first two chunks of weights.  A barrier after global-to-LDS copies waits
    // for every outstanding load, so the remaining chunks are issued after it
    // (with their share of the row scaling).
    {
      const int cpr = d / 8;  // 16-byte chunks per row
      for (int r = ld; r < nt + (FOLD ? 0 : 1); r += NW - 1) {  // rows, then gamma
        const int nb = (n0 + r) / a.T, ntk = n0 + r - nb * a.T;
        const uint16_t* src = (r < nt ? static_cast<const uint16_t*>(a.h) + ((size_t)nb * a.h_ld + ntk) * d
                                      : static_cast<const uint16_t*>(a.gamma)) + 8 * lane;
        uint16_t* dst = r < nt ? hb + (size_t)r * HLD : gl;
        for (int ch0 = 0; ch0 < cpr; ch0 += 64)
          if (ch0 + lane < cpr)
            __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(src + 8 * ch0),
                                             (__attribute__((address_space(3))) void*)(dst + 8 * ch0), 16, 0, 0);
      }
    }
    load_chunk(wr[0], 0);
    if (1 < nchunks) load_chunk(wr[1], 1);
    __syncthreads();
#pragma unroll
    for (int u = 2; u < D; ++u)
      if (u < nchunks) load_chunk(wr[u], u);
    scale_rows();
    store_chunk(wr[0], 0);
    if (D < nchunks) load_chunk(wr[0], D);
    __syncthreads();
    // sums of squares: row 8 ld + (lane >> 3), column chunk lane & 7, K-steps in
    // order (the tile engine's per-thread chain), one chunk of K-steps per
    // iteration; the 8 lanes' sums by the xor tree and 1/rms before the last barrier
    const int srow = 8 * ld + (lane >> 3), sub = lane & 7;
    const uint16_t* hr = hb + (size_t)(srow < nt ? srow : 0) * HLD + 8 * sub;
    float ss = 0.0f;
    uint4 xs[CK];  // the next chunk's residual values, read one iteration ahead
    auto ss_read = [&](int c) {
#pragma unroll
      for (int kk = 0; kk < CK; ++kk) xs[kk] = *reinterpret_cast<const uint4*>(hr + (size_t)min(c * CK + kk, nsteps - 1) * kKT);
    };
    auto ss_chunk = [&](int c) {
      uint4 x[CK];
#pragma unroll
      for (int kk = 0; kk < CK; ++kk) x[kk] = xs[kk];
      if (c + 1 < nchunks) ss_read(c + 1);
      if (srow < nt) {
#pragma unroll
        for (int kk = 0; kk < CK; ++kk)
          if (c * CK + kk < nsteps) sumsq_chunk<FOLD>(x[kk], ss);
      }
    };
    ss_read(0);
    auto finish_ss = [&]() {
      ss += __shfl_xor(ss, 1, 64);
      ss += __shfl_xor(ss, 2, 64);
      ss += __shfl_xor(ss, 4, 64);
      if (sub == 0 && srow < kProjTok) rinv[srow] = srow < nt ? 1.0f / sqrtf(ss / (float)d + a.eps) : 0.0f;
    };
    // iteration c: the sums of squares of chunk c, write chunk c + 1 (loaded D
    // chunks earlier), refill its registers with chunk c + 1 + D, barrier c
    if constexpr (NCH > 0) {
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        ss_chunk(c);
        if (c + 1 < NCH) {
          store_chunk(wr[(c + 1) % D], c + 1);
          if (c + 1 + D < NCH) load_chunk(wr[(c + 1) % D], c + 1 + D);
        } else {
          finish_ss();
        }
        __syncthreads();
      }
    } else {
      for (int c0 = 0; c0 < nchunks; c0 += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) {
          const int c = c0 + u;
          if (c < nchunks) {
            ss_chunk(c);
            if (c + 1 < nchunks) {
              store_chunk(wr[(u + 1) % D], c + 1);
              if (c + 1 + D < nchunks) load_chunk(wr[(u + 1) % D], c + 1 + D);
            } else {
              finish_ss();
            }
            __syncthreads();
          }
        }
      }
    }
    return;
  }

  // wave 0: the RoPE table and positions, then its share of gamma * h (while the
  // loaders issue their weights and scale theirs), then the MFMA chain
  for (int i = lane; i < HD / 2; i += 64) rev[i] = a.rev[i];
  if (lane < kProjTok) {
    const int nb = (n0 + lane) / a.T, ntk = n0 + lane - nb * a.T;
    pos[lane] = lane < nt ? a.pos0[nb] + ntk : 0;
  }
  __syncthreads();
  scale_rows();
  __syncthreads();
  // MFMA over d: A = 32 weight rows (from the ring), B = the group's tokens.
  // Columns of absent tokens read row 0 and hold unused values: MFMA output
  // columns are independent and only those of present tokens are stored.
  const int col = lane & 31;
  const uint16_t* hcol = (FOLD ? hb : hs) + (size_t)(col < nt ? col : 0) * HLD + 8 * (lane >> 5);
  {
    bf16x8_t a0[FPC], b0f[FPC], a1[FPC], b1f[FPC];  // chunk c's fragments and chunk c + 1's
    auto read_chunk = [&](bf16x8_t (&av)[FPC], bf16x8_t (&bv)[FPC], int c) {
      const uint16_t* slot = ring + (size_t)(c % NR) * FPC * 512 + 8 * lane;
#pragma unroll
      for (int f = 0; f < FPC; ++f) {
        const int s = min(c * CK + (f >> 2), nsteps - 1);
        av[f] = *reinterpret_cast<const bf16x8_t*>(slot + f * 512);
        bv[f] = *reinterpret_cast<const bf16x8_t*>(hcol + (size_t)s * kKT + 16 * (f & 3));
      }
    };
    auto step = [&](int c, bf16x8_t (&ac)[FPC], bf16x8_t (&bc)[FPC], bf16x8_t (&an)[FPC], bf16x8_t (&bn)[FPC]) {
      __syncthreads();
      if (c + 1 < nchunks) read_chunk(an, bn, c + 1);
      const int nk = min(CK, nsteps - c * CK);
#pragma unroll
      for (int f = 0; f < FPC; ++f)
        if ((f >> 2) < nk) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ac[f], bc[f], acc, 0, 0, 0);
    };
    read_chunk(a0, b0f, 0);
    for (int c = 0; c < nchunks; c += 2) {
      step(c, a0, b0f, a1, b1f);
      if (c + 1 < nchunks) step(c + 1, a1, b1f, a0, b0f);
    }
  }

  if (col >= nt) return;
  const float ri = rinv[col];
  const int p = pos[col];
  const int b = (n0 + col) / a.T, t = n0 + col - b * a.T;
  float v[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) v[r] = acc[r] * ri;
  const int head = row0 / HD, f0 = row0 % HD;
  if (rope) {
#pragma unroll
    for (int r = 0; r < 16; r += 2) {
      const int f = f0 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      rope_rotate(v[r], v[r + 1], p, rev[f >> 1]);
    }
  }
  uint16_t* dst;
  if (mat == 0) {
    dst = static_cast<uint16_t*>(a.q_out) + ((size_t)b * a.n_q + head) * HD;
  } else {
    uint16_t* base = static_cast<uint16_t*>(mat == 1 ? a.k_out : a.v_out);
    dst = base + (((size_t)b * a.n_kv + head) * a.kv_t_cap + a.kv_t_off + t) * HD;
  }
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    const int f = f0 + 8 * g4 + 4 * (lane >> 5);
    uint2 o;
    o.x = pack_bf16x2(v[4 * g4 + 0], v[4 * g4 + 1]);
    o.y = pack_bf16x2(v[4 * g4 + 2], v[4 * g4 + 3]);
    *reinterpret_cast<uint2*>(dst + f) = o;
  }
}

// ------------------------------------------------------------------ fused recompute + attention

// grid: xcd_map(n_kv * B * C) workgroups, one per (KV head j, sequence b, chunk c),
// C = n_tail + n_rec.  Chunks c < n_tail attend stored tail tile c (64 rows, the
// last one up to 64 + fold_rows<T>(); partial n_rec + c) and come first, as they
// are short; chunk n_tail + r recomputes residual rows r*MT..r*MT+MT-1 (partial
// r).  A folded tail (<= fold_rows<T>() rows, n_tail = 0) is attended with the
// last recomputed chunk's keys.  MT = kMtWide: the wide engine (bf16, 128-key
// chunks).
template <typename T, int HD, int MT, bool PACKED, bool FOLD>
__device__ __forceinline__ void fused_body(const FusedArgs& a, int per_xcd, int hg) {
  extern __shared__ __align__(16) char lds[];
  constexpr bool WIDE = MT == kMtWide;
  constexpr int NT = WIDE ? kNtWide : kNtTile;
  constexpr int FR = fold_rows<T>();
  constexpr ProjLds PL = proj_lds<T>(HD, MT, FR);
  constexpr int CPT = MT * 8 / NT;
  constexpr int KLD = kv_ld<T>(HD);
  constexpr int KPL = (MT + FR + 63) / 64;  // keys per lane of the tile attention
  static_assert(MT == kTile || (WIDE && sizeof(T) == 2), "fused chunks: 64-key tiles, or the wide bf16 engine");
  const int tid = threadIdx.x;
  const bool fold = fold_tail<T>(a.n_rec, a.T_tail);
  const int n_tail = fused_tail_tiles<T>(a.n_rec, a.T_tail);
  const int C = n_tail + a.n_rec;
  // 32-bit index arithmetic (the item count is below 2^31, checked by the host):
  // every wave runs it on the CU's one scalar unit before its first load.
  const unsigned item = (blockIdx.x % kXcds) * (unsigned)per_xcd + blockIdx.x / kXcds;
  if (item >= (unsigned)a.n_kv * (unsigned)a.B * (unsigned)C) return;
  // Items in XCD order: KV heads in groups of hg (a power of two dividing n_kv) of
  // one sequence, the group's chunks in order, its heads alternating.  An XCD's
  // run of per_xcd items then spans hg heads and per_xcd / hg chunks; it pulls
  // each of those residual tiles and each of those heads' weights into its own
  // L2 once.  The host picks hg to balance the two streams (fused_head_group).
  const int hg_log2 = __builtin_ctz((unsigned)hg);
  const unsigned hgC = (unsigned)C << hg_log2;
  const unsigned gi = item / hgC, rem = item - gi * hgC;  // group index jg * B + b
  const int jg = (int)(gi / (unsigned)a.B);
  const int b = (int)(gi - (unsigned)jg * (unsigned)a.B);
  const int c = (int)(rem >> hg_log2);
  const int j = (jg << hg_log2) + (int)(rem & (unsigned)(hg - 1));
  const int rc = c - n_tail;  // recomputed chunk (c >= n_tail)
  const int g = a.n_q / a.n_kv;
  const AttnLds AL = attn_lds(PL.end, g, HD, MT + FR);
  T* kv = reinterpret_cast<T*>(lds + PL.kv);

  // A folded tail goes to the last recomputed tile's workgroup: its rows are
  // loaded with the setup values (one 16-byte chunk of a K | V row per thread;
  // other threads load q, which is always readable) and land in LDS rows MT..
  // while the tile is being recomputed.
  const bool tail_here = fold && rc == a.n_rec - 1;
  constexpr int TCH = 2 * HD * (int)sizeof(T) / 16;  // chunks per K | V row
  static_assert(FR * TCH <= NT, "one folded-tail chunk per thread");
  const int tr = tid / TCH, tch = tid - tr * TCH;
  const bool tail_mine = FR > 0 && tail_here && tr < a.T_tail;
  u32x4_t tail_v;
  if constexpr (FR > 0) {
    int tslot = a.tail_t_off + (tail_mine ? tr : 0);  // tail rows wrap around a ring of tail_t_cap slots
    tslot -= tslot >= a.tail_t_cap ? a.tail_t_cap : 0;
    const size_t trow = ((size_t)b * a.n_kv + j) * a.tail_t_cap + tslot;
    const T* src = tch < TCH / 2 ? static_cast<const T*>(a.tk) + trow * HD + tch * (16 / sizeof(T))
                                 : static_cast<const T*>(a.tv) + trow * HD + (tch - TCH / 2) * (16 / sizeof(T));
    tail_v = *reinterpret_cast<const u32x4_t*>(tail_mine ? src : static_cast<const T*>(a.q));
  }

  if (c >= n_tail) {
    const int t0 = rc * MT;
    const int n = min(MT, a.T_rec - t0);
    double* rev = reinterpret_cast<double*>(lds + PL.rev);
    float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
    int* pos = reinterpret_cast<int*>(lds + PL.pos);
    T* hst = reinterpret_cast<T*>(lds + PL.hst);
    uint16_t* gam = reinterpret_cast<uint16_t*>(lds + AL.end);
    // q, gamma and rev reach LDS while the K-loop's first loads are in flight
    const TileSetup<T, HD, NT, true, !FOLD> su(static_cast<const T*>(a.q), b, a.n_q, j, g, a.gamma, a.d, a.rev);
    // pos0[b] is read here, after the K-loop's first loads are issued: a scalar
    // load read up front holds back every address computation behind its latency
    auto setup = [&]() {
      const int p0 = (a.pos0 != nullptr ? a.pos0[b] : 0) + t0;
      su.store(reinterpret_cast<float*>(lds + AL.q), gam, rev);
      if (tid < MT) pos[tid] = p0 + tid;
      if constexpr (FR > 0) {
        if (tail_mine) *reinterpret_cast<u32x4_t*>(kv + (size_t)(MT + tr) * KLD + tch * (16 / sizeof(T))) = tail_v;
      }
    };
    const T* hrow[CPT];
    bool valid[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
      const int t = (tid >> 3) + (NT / 8) * r;
      valid[r] = t < n;
      hrow[r] = static_cast<const T*>(a.h) + ((size_t)b * a.h_ld + t0 + (valid[r] ? t : 0)) * a.d + 8 * (tid & 7);
    }
    const size_t hd_d = (size_t)HD * a.d;
    const Half halves[2] = {Half{static_cast<const T*>(a.w_k) + j * hd_d, 1},
                            Half{static_cast<const T*>(a.w_v) + j * hd_d, 0}};
    if constexpr (sizeof(T) == 2 && HD >= 128) {
      // residual rows two K-steps ahead on 64-token tiles (RLEAD), one on the wide engine
      WideTile<HD, MT, PACKED, FOLD, kNtWide, kv_ld<uint16_t>(HD), false, MT == 64>::run(
          static_cast<const uint16_t*>(a.h) + ((size_t)b * a.h_ld + t0) * a.d, n, gam,
          static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves, hst, rinv, pos, rev, kv, setup);
    } else if constexpr (sizeof(T) == 2) {
      MfmaTile<HD, MT, PACKED, FOLD>::run(hrow, valid, gam, static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves,
                                          hst, rinv, pos, rev, kv, setup);
    } else {
      F32Tile<HD, MT>::run(hrow, valid, static_cast<const float*>(a.gamma), a.d, a.eps, halves, hst, rinv, pos, rev,
                           kv, setup);
    }
    __syncthreads();
    if (a.dbg_k != nullptr) {
      constexpr int CH = 16 / sizeof(T);
      constexpr int CPR = HD / CH;
      for (int i = tid; i < 2 * n * CPR; i += NT) {
        const int half = i / (n * CPR);
        const int rem = i - half * n * CPR;
        const int row = rem / CPR, ch = rem - row * CPR;
        T* base = static_cast<T*>(half ? a.dbg_v : a.dbg_k);
        T* dst = base + (((size_t)b * a.n_kv + j) * a.dbg_t_cap + a.dbg_t_off + t0 + row) * HD;
        *reinterpret_cast<uint4*>(dst + ch * CH) =
            *reinterpret_cast<const uint4*>(kv + (size_t)row * KLD + half * HD + ch * CH);
      }
    }
    int nk = n;
    if constexpr (FR > 0) {
      if (tail_here) {
        if (n < MT) move_rows<T, HD, NT, FR>(kv, MT, n, a.T_tail);
        nk = n + a.T_tail;
      }
    }
    attend_tile<T, HD, NT, KPL>(kv, nk, MT + FR, g, lds, AL);
    write_partial<HD, NT>(lds, AL, a.ws_acc, a.ws_ml, b, a.n_q, j, g, a.S, rc, tile_splits<T>(g));
  } else {
    // tail tile c: 64 rows, the last one the rest (up to 64 + FR rows)
    const int r0 = c * kTile;
    const int nk = c == n_tail - 1 ? a.T_tail - r0 : kTile;
    load_q<T, HD, NT>(static_cast<const T*>(a.q), b, a.n_q, j, g, reinterpret_cast<float*>(lds + AL.q));
    int tr0 = a.tail_t_off + r0;  // the ring's slot of row r0 (a ring of tail_t_cap slots)
    tr0 -= tr0 >= a.tail_t_cap ? a.tail_t_cap : 0;
    load_kv_tile<T, HD, NT>(static_cast<const T*>(a.tk), static_cast<const T*>(a.tv), b, a.n_kv, j, a.tail_t_cap,
                            tr0, min(nk, kTile), kv);
    if (nk > kTile) {
      int tr1 = tr0 + kTile;
      tr1 -= tr1 >= a.tail_t_cap ? a.tail_t_cap : 0;
      load_kv_tile<T, HD, NT>(static_cast<const T*>(a.tk), static_cast<const T*>(a.tv), b, a.n_kv, j, a.tail_t_cap,
                              tr1, nk - kTile, kv + (size_t)kTile * KLD);
    }
    __syncthreads();
    attend_tile<T, HD, NT, KPL>(kv, nk, MT + FR, g, lds, AL);
    write_partial<HD, NT>(lds, AL, a.ws_acc, a.ws_ml, b, a.n_q, j, g, a.S, a.n_rec + c, tile_splits<T>(g));
  }
  if (a.out != nullptr) {
    unsigned long long* ctr = a.ws_done + (size_t)b * a.n_kv + j;
    const unsigned long long before = split_arrive(ctr, 1, reinterpret_cast<unsigned long long*>(lds + AL.ctr));
    if (split_complete(ctr, before, 1, a.S))
      combine_rows<T, HD, NT>(a.ws_acc, a.ws_ml, static_cast<T*>(a.out), (size_t)b * a.n_q + (size_t)j * g, g, a.S,
                              reinterpret_cast<float*>(lds + AL.cmb));
  }
}

template <typename T, int HD, int MT, bool PACKED, bool FOLD>
__global__ __launch_bounds__(kNtTile, 1) void fused_kernel(FusedArgs a, int per_xcd, int hg) {
  fused_body<T, HD, MT, PACKED, FOLD>(a, per_xcd, hg);
}

// One workgroup of 8 waves per CU, two per SIMD: 256 registers per lane (the
// wave's 128-token accumulators in AGPRs).
template <int HD, bool PACKED, bool FOLD>
__global__ __launch_bounds__(kNtWide, 1) void fused_wide_kernel(
    FusedArgs a, int per_xcd, int hg) {
  fused_body<uint16_t, HD, kMtWide, PACKED, FOLD>(a, per_xcd, hg);
}

// ------------------------------------------------------------------ fused recompute + attention, KV-head pairs

// bf16, head_dim 128: one workgroup per (pair of KV heads 2 jp, 2 jp + 1,
// sequence b, chunk c) on the wide engine's head_dim 256 wave layout.  The K
// rows of both heads are the tile's 256 "K" rows and their V rows its 256 "V"
// rows (the heads' rows are adjacent in W_k / W_v), so each wave runs two
// 32-row blocks for all four token blocks and every residual B fragment read
// from LDS feeds twice the MFMAs of the head_dim 128 wide tile.  Per element
// the MFMA chain over d, 1/rms and the RoPE epilogue are the wide engine's, and
// the RoPE table holds head_dim 128's 64 frequencies twice (rows 128.. of a
// half are the second head's features 0..), so K/V equal every other engine's
// bit for bit.  The K|V tile row is [K head 0 | K head 1 | V head 0 | V head
// 1]; the attention, partial, arrival and merge then run per head, as on the
// wide engine, with both groups' q rows in LDS.  Chunks c < n_tail attend the
// stored tail tiles of both heads, one after the other.
template <bool PACKED, bool FOLD>
__global__ __launch_bounds__(kNtWide, 1) void fused_pair_kernel(FusedArgs a, int per_xcd, int hg) {
  extern __shared__ __align__(16) char lds[];
  constexpr int HD = 128, MT = kMtWide, NT = kNtWide;
  constexpr int FR = fold_rows<uint16_t>();
  constexpr ProjLds PL = proj_lds<uint16_t>(2 * HD, MT, FR);
  constexpr int KLD = kv_ld<uint16_t>(2 * HD);  // pair tile row stride
  constexpr int KPL = (MT + FR + 63) / 64;
  const int tid = threadIdx.x;
  const bool fold = fold_tail<uint16_t>(a.n_rec, a.T_tail);
  const int n_tail = fused_tail_tiles<uint16_t>(a.n_rec, a.T_tail);
  const int C = n_tail + a.n_rec;
  const int np = a.n_kv >> 1;
  const unsigned item = (blockIdx.x % kXcds) * (unsigned)per_xcd + blockIdx.x / kXcds;
  if (item >= (unsigned)np * (unsigned)a.B * (unsigned)C) return;
  // items as on the wide engine, with head pairs in place of heads
  const int hg_log2 = __builtin_ctz((unsigned)hg);
  const unsigned hgC = (unsigned)C << hg_log2;
  const unsigned gi = item / hgC, rem = item - gi * hgC;
  const int pg = (int)(gi / (unsigned)a.B);
  const int b = (int)(gi - (unsigned)pg * (unsigned)a.B);
  const int c = (int)(rem >> hg_log2);
  const int jp = (pg << hg_log2) + (int)(rem & (unsigned)(hg - 1));
  const int j0 = 2 * jp;  // first KV head of the pair
  const int rc = c - n_tail;
  const int g = a.n_q / a.n_kv;
  const AttnLds AL = attn_lds(PL.end, g, HD, MT + FR);
  uint16_t* kv = reinterpret_cast<uint16_t*>(lds + PL.kv);
  // LDS of head hh's attention: its group's q rows follow the first group's
  auto head_lds = [&](int hh) {
    AttnLds L = AL;
    L.q = AL.q + (size_t)hh * g * HD * sizeof(uint16_t);
    return L;
  };
  const uint16_t* const tk = static_cast<const uint16_t*>(a.tk);
  const uint16_t* const tv = static_cast<const uint16_t*>(a.tv);

  // folded tail: one 16-byte chunk of a pair row per thread (64 chunks a row),
  // copied into LDS rows MT.. by the tile's setup
  const bool tail_here = fold && rc == a.n_rec - 1;
  constexpr int TCH = 4 * HD * 2 / 16;
  static_assert(FR * TCH <= NT, "one folded-tail chunk per thread");

  if (c >= n_tail) {
    const int t0 = rc * MT;
    const int n = min(MT, a.T_rec - t0);
    double* rev = reinterpret_cast<double*>(lds + PL.rev);
    float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
    int* pos = reinterpret_cast<int*>(lds + PL.pos);
    uint16_t* hst = reinterpret_cast<uint16_t*>(lds + PL.hst);
    uint16_t* gam = reinterpret_cast<uint16_t*>(lds + AL.end);
    // both groups' q rows (2 g heads from head j0 * g), gamma, the 64 frequencies
    const TileSetup<uint16_t, HD, NT, true, !FOLD> su(static_cast<const uint16_t*>(a.q), b, a.n_q, jp, 2 * g,
                                                      a.gamma, a.d, a.rev);
    auto setup = [&]() {
      const int p0 = (a.pos0 != nullptr ? a.pos0[b] : 0) + t0;
      su.store(reinterpret_cast<float*>(lds + AL.q), gam, rev);
      if (tid >= HD / 2 && tid < HD) rev[tid] = a.rev[tid - HD / 2];  // frequency f % 64 at f
      if (tid < MT) pos[tid] = p0 + tid;
      const int tr = tid / TCH, tch = tid - tr * TCH;
      if (tail_here && tr < a.T_tail) {
        int tslot = a.tail_t_off + tr;
        tslot -= tslot >= a.tail_t_cap ? a.tail_t_cap : 0;
        const int part = tch >> 4;  // K head 0, K head 1, V head 0, V head 1
        const size_t trow = ((size_t)b * a.n_kv + j0 + (part & 1)) * a.tail_t_cap + tslot;
        *reinterpret_cast<u32x4_t*>(kv + (size_t)(MT + tr) * KLD + 8 * tch) =
            *reinterpret_cast<const u32x4_t*>((part >= 2 ? tv : tk) + trow * HD + 8 * (tch & 15));
      }
    };
    const size_t hd_d = (size_t)HD * a.d;
    const Half halves[2] = {Half{static_cast<const uint16_t*>(a.w_k) + j0 * hd_d, 1},
                            Half{static_cast<const uint16_t*>(a.w_v) + j0 * hd_d, 0}};
    WideTile<2 * HD, MT, PACKED, FOLD, NT, KLD, false, true>::run(static_cast<const uint16_t*>(a.h) + ((size_t)b * a.h_ld + t0) * a.d, n,
                                            gam, static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves, hst, rinv,
                                            pos, rev, kv, setup);
    __syncthreads();
    if (a.dbg_k != nullptr) {
      constexpr int CPR = HD / 8;
      for (int i = tid; i < 4 * n * CPR; i += NT) {
        const int part = i / (n * CPR);
        const int r2 = i - part * n * CPR;
        const int row = r2 / CPR, ch = r2 - row * CPR;
        uint16_t* base = static_cast<uint16_t*>(part >= 2 ? a.dbg_v : a.dbg_k);
        uint16_t* dst = base + (((size_t)b * a.n_kv + j0 + (part & 1)) * a.dbg_t_cap + a.dbg_t_off + t0 + row) * HD;
        *reinterpret_cast<uint4*>(dst + 8 * ch) = *reinterpret_cast<const uint4*>(kv + (size_t)row * KLD + part * HD + 8 * ch);
      }
    }
    int nk = n;
    if (tail_here) {
      if (n < MT) move_rows<uint16_t, 2 * HD, NT, FR>(kv, MT, n, a.T_tail);
      nk = n + a.T_tail;
    }
    for (int hh = 0; hh < 2; ++hh) {
      const AttnLds L = head_lds(hh);
      attend_scores_mfma<HD, NT, KPL, KLD>(kv + hh * HD, nk, MT + FR, g, lds, L);
      attend_pv_mfma<HD, NT, KLD>(kv + (2 + hh) * HD, nk, MT + FR, g, lds, L);
      write_partial<HD, NT>(lds, L, a.ws_acc, a.ws_ml, b, a.n_q, j0 + hh, g, a.S, rc, 1);
      __syncthreads();
    }
  } else {
    // tail tile c of each head in turn, on the head_dim 128 tile layout
    const int r0 = c * kTile;
    const int nk = c == n_tail - 1 ? a.T_tail - r0 : kTile;
    load_q<uint16_t, HD, NT>(static_cast<const uint16_t*>(a.q), b, a.n_q, jp, 2 * g,
                             reinterpret_cast<float*>(lds + AL.q));
    int tr0 = a.tail_t_off + r0;
    tr0 -= tr0 >= a.tail_t_cap ? a.tail_t_cap : 0;
    int tr1 = tr0 + kTile;
    tr1 -= tr1 >= a.tail_t_cap ? a.tail_t_cap : 0;
    for (int hh = 0; hh < 2; ++hh) {
      load_kv_tile<uint16_t, HD, NT>(tk, tv, b, a.n_kv, j0 + hh, a.tail_t_cap, tr0, min(nk, kTile), kv);
      if (nk > kTile)
        load_kv_tile<uint16_t, HD, NT>(tk, tv, b, a.n_kv, j0 + hh, a.tail_t_cap, tr1, nk - kTile,
                                       kv + (size_t)kTile * kv_ld<uint16_t>(HD));
      __syncthreads();
      const AttnLds L = head_lds(hh);
      attend_tile<uint16_t, HD, NT, KPL>(kv, nk, MT + FR, g, lds, L);
      write_partial<HD, NT>(lds, L, a.ws_acc, a.ws_ml, b, a.n_q, j0 + hh, g, a.S, a.n_rec + c, 1);
      __syncthreads();
    }
  }
  if (a.out != nullptr) {
    // arrivals at both heads' counters, then one merge of the rows of the heads
    // this workgroup completed (rows are merged independently of each other)
    bool last[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      unsigned long long* ctr = a.ws_done + (size_t)b * a.n_kv + j0 + hh;
      const unsigned long long before = split_arrive(ctr, 1, reinterpret_cast<unsigned long long*>(lds + AL.ctr));
      last[hh] = split_complete(ctr, before, 1, a.S);
    }
    const int first = last[0] ? 0 : 1;
    const int cnt = (int)last[0] + (int)last[1];
    if (cnt > 0)
      combine_rows<uint16_t, HD, NT>(a.ws_acc, a.ws_ml, static_cast<uint16_t*>(a.out),
                                     (size_t)b * a.n_q + (size_t)(j0 + first) * g, cnt * g, a.S,
                                     reinterpret_cast<float*>(lds + AL.cmb));
  }
}

// ------------------------------------------------------------------ fused recompute + attention, split engine

// bf16, head_dim 128 / 256, for calls with too few 128-token tiles to fill the
// chip with both halves per workgroup.  Per (KV head j, sequence b, 128-token
// chunk c) two workgroups of split_nt(HD) threads on the split engine: the K
// role recomputes the chunk's K rows (with RoPE) and takes tasks 1-2 of the
// tile attention (scores, max, sum, probabilities), which it writes to the
// chunk's exchange record before setting bit c of the (b, j) completion words;
// the V role recomputes the V rows, waits for that bit (a bounded wait), reads
// the record and takes task 3 (P V), then writes the chunk's split-K partial,
// arrives at the (b, j) counter and, if last, merges.  The K role of a pair is
// the item before its V role, on the same XCD, so it is dispatched no later
// than the V role that waits for it and depends on nothing itself.  A folded
// tail (T_tail <= fold rows: the current token) joins the last chunk, its K
// rows in the K role's tile and its V rows in the V role's.  grid:
// xcd_map(2 * n_kv * B * n_rec), items ordered as fused_body's chunks.
template <int HD, int MT, bool PACKED, bool FOLD>
__global__ __launch_bounds__(split_nt(HD), 1) void fused_split_kernel(FusedArgs a, int per_xcd, int hg) {
  extern __shared__ __align__(16) char lds[];
  constexpr int NT = split_nt(HD), FR = fold_rows<uint16_t>();
  constexpr int KPL = (MT + FR + 63) / 64;  // keys per lane of the tile attention
  constexpr ProjLds PL = split_lds(HD, MT, FR);
  constexpr int KLD = split_ld(HD);
  constexpr int CPR = HD / 8;  // 16-byte chunks of a K (or V) row
  static_assert(FR * CPR <= NT, "one folded-tail chunk per thread");
  const int tid = threadIdx.x;
  const int C = a.n_rec;
  const unsigned item = (blockIdx.x % kXcds) * (unsigned)per_xcd + blockIdx.x / kXcds;
  if (item >= 2u * (unsigned)a.n_kv * (unsigned)a.B * (unsigned)C) return;
  const int role = (int)(item & 1u);  // 0: K rows, 1: V rows
  const unsigned pair = item >> 1;
  const int hg_log2 = __builtin_ctz((unsigned)hg);
  const unsigned hgC = (unsigned)C << hg_log2;
  const unsigned gi = pair / hgC, rem = pair - gi * hgC;
  const int jg = (int)(gi / (unsigned)a.B);
  const int b = (int)(gi - (unsigned)jg * (unsigned)a.B);
  const int c = (int)(rem >> hg_log2);
  const int j = (jg << hg_log2) + (int)(rem & (unsigned)(hg - 1));
  const int g = a.n_q / a.n_kv;
  constexpr int ROWS = MT + FR;
  const AttnLds AL = attn_lds(PL.end, g, HD, ROWS);
  uint16_t* tile = reinterpret_cast<uint16_t*>(lds + PL.kv);
  const int t0 = c * MT;
  const int n = min(MT, a.T_rec - t0);

  // folded tail rows of this role's half, loaded with the setup values
  const bool tail_here = a.T_tail > 0 && c == C - 1;
  const int tr = tid / CPR, tch = tid - tr * CPR;
  const bool tail_mine = tail_here && tr < a.T_tail;
  u32x4_t tail_v;
  {
    int tslot = a.tail_t_off + (tail_mine ? tr : 0);  // a ring of tail_t_cap slots
    tslot -= tslot >= a.tail_t_cap ? a.tail_t_cap : 0;
    const size_t trow = ((size_t)b * a.n_kv + j) * a.tail_t_cap + tslot;
    const uint16_t* src = static_cast<const uint16_t*>(role ? a.tv : a.tk) + trow * HD + tch * 8;
    tail_v = *reinterpret_cast<const u32x4_t*>(tail_mine ? src : static_cast<const uint16_t*>(a.q));
  }

  double* rev = reinterpret_cast<double*>(lds + PL.rev);
  float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
  int* pos = reinterpret_cast<int*>(lds + PL.pos);
  uint16_t* hst = reinterpret_cast<uint16_t*>(lds + PL.hst);
  uint16_t* gam = reinterpret_cast<uint16_t*>(lds + AL.end);
  const TileSetup<uint16_t, HD, NT, true, !FOLD> su(static_cast<const uint16_t*>(a.q), b, a.n_q, j, g, a.gamma, a.d,
                                                     a.rev);
  auto setup = [&]() {
    const int p0 = (a.pos0 != nullptr ? a.pos0[b] : 0) + t0;
    su.store(reinterpret_cast<float*>(lds + AL.q), gam, rev);
    if (tid < MT) pos[tid] = p0 + tid;
    if (tail_mine) *reinterpret_cast<u32x4_t*>(tile + (size_t)(MT + tr) * KLD + tch * 8) = tail_v;
  };
  const size_t hd_d = (size_t)HD * a.d;
  const Half halves[2] = {Half{static_cast<const uint16_t*>(role ? a.w_v : a.w_k) + j * hd_d, 1 - role},
                          Half{nullptr, 0}};
  WideTile<HD, MT, PACKED, FOLD, NT, KLD, true>::run(static_cast<const uint16_t*>(a.h) + ((size_t)b * a.h_ld + t0) * a.d,
                                                     n, gam, static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves,
                                                     hst, rinv, pos, rev, tile, setup);
  __syncthreads();
  if (a.dbg_k != nullptr) {
    uint16_t* base = static_cast<uint16_t*>(role ? a.dbg_v : a.dbg_k);
    uint16_t* dst = base + (((size_t)b * a.n_kv + j) * a.dbg_t_cap + a.dbg_t_off + t0) * HD;
    for (int i = tid; i < n * CPR; i += NT) {
      const int row = i / CPR, ch = i - row * CPR;
      *reinterpret_cast<uint4*>(dst + (size_t)row * HD + ch * 8) =
          *reinterpret_cast<const uint4*>(tile + (size_t)row * KLD + ch * 8);
    }
  }
  int nk = n;
  if (tail_here) {
    if (n < MT) move_rows<uint16_t, HD, NT, FR, HD, KLD>(tile, MT, n, a.T_tail);
    nk = n + a.T_tail;
  }
  float* S = reinterpret_cast<float*>(lds + AL.s);
  float* ml = reinterpret_cast<float*>(lds + AL.ml);
  float* xrec = a.xch + (((size_t)b * a.n_kv + j) * C + c) * a.xf;
  unsigned long long* bits = a.ws_bits + ((size_t)b * a.n_kv + j) * kSplitBitWords;
  if (role == 0) {
    attend_scores_mfma<HD, NT, KPL, KLD>(tile, nk, ROWS, g, lds, AL);
    for (int i = tid; i < g * ROWS; i += NT) store_dev(xrec + i, S[i]);
    if (tid < 2 * g) store_dev(xrec + g * ROWS + tid, ml[tid]);
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this thread's record stores are complete
    __syncthreads();
    if (tid == 0)
      __hip_atomic_fetch_or(bits + (c >> 6), 1ull << (c & 63), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  int* flag = reinterpret_cast<int*>(lds + AL.ctr);
  if (tid == 0) {
    int ok = 0;
    for (unsigned it = 0; it < kSplitSpinLimit; ++it) {
      if ((__hip_atomic_load(bits + (c >> 6), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >> (c & 63)) & 1ull) {
        ok = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    *flag = ok;
  }
  __syncthreads();
  const bool ok = *flag != 0;
  for (int i = tid; i < g * ROWS; i += NT) S[i] = load_dev(xrec + i);
  if (tid < 2 * g) ml[tid] = ok ? load_dev(xrec + g * ROWS + tid) : __builtin_nanf("");
  __syncthreads();
  attend_pv_mfma<HD, NT, KLD>(tile, nk, ROWS, g, lds, AL);
  write_partial<HD, NT>(lds, AL, a.ws_acc, a.ws_ml, b, a.n_q, j, g, a.S, c, tile_splits<uint16_t>(g));
  // every V role arrives (also without out): the last one clears the
  // completion words for the next call
  unsigned long long* ctr = a.ws_done + (size_t)b * a.n_kv + j;
  const unsigned long long before = split_arrive(ctr, 1, reinterpret_cast<unsigned long long*>(lds + AL.ctr));
  if (split_complete(ctr, before, 1, a.S)) {
    if (tid < kSplitBitWords) __hip_atomic_store(bits + tid, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (a.out != nullptr)
      combine_rows<uint16_t, HD, NT>(a.ws_acc, a.ws_ml, static_cast<uint16_t*>(a.out),
                                     (size_t)b * a.n_q + (size_t)j * g, g, a.S, reinterpret_cast<float*>(lds + AL.cmb));
  }
}

// ------------------------------------------------------------------ stored-K/V attention

template <typename T, int HD>
__global__ __launch_bounds__(kNtAttn) void decode_kernel(AttnArgs a) {
  extern __shared__ __align__(16) char lds[];
  constexpr int NT = kNtAttn;
  const int s = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int g = a.n_q / a.n_kv;
  constexpr int FR = fold_rows<T>();
  const AttnLds AL = attn_lds(align_up(sizeof(T) * (kTile + FR) * kv_ld<T>(HD), 16), g, HD, kTile + FR);
  T* kv = reinterpret_cast<T*>(lds);
  const int t0 = s * kTile;
  const int n = s == a.S - 1 ? a.T - t0 : kTile;  // the last tile may hold a folded remainder
  if constexpr (FR > 0) {
    if (n > kTile)
      prefetch_rows_lds<T, HD>(static_cast<const T*>(a.k), static_cast<const T*>(a.v),
                               ((size_t)b * a.n_kv + j) * a.t_cap + a.t_off + t0 + kTile, n - kTile,
                               kv + (size_t)kTile * kv_ld<T>(HD));
  }
  load_kv_tile<T, HD, NT>(static_cast<const T*>(a.k), static_cast<const T*>(a.v), b, a.n_kv, j, a.t_cap,
                          a.t_off + t0, min(n, kTile), kv);
  load_q<T, HD, NT>(static_cast<const T*>(a.q), b, a.n_q, j, g, reinterpret_cast<float*>(lds + AL.q));
  if constexpr (FR > 0) __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): the remainder rows are in LDS
  __syncthreads();
  attend_tile<T, HD, NT, tile_kpl<T>()>(kv, n, kTile + FR, g, lds, AL);
  write_partial<HD, NT>(lds, AL, a.ws_acc, a.ws_ml, b, a.n_q, j, g, a.S, s, tile_splits<T>(g));
  if (a.out != nullptr) {
    unsigned long long* ctr = a.ws_done + (size_t)b * a.n_kv + j;
    const unsigned long long before = split_arrive(ctr, 1, reinterpret_cast<unsigned long long*>(lds + AL.ctr));
    if (split_complete(ctr, before, 1, a.S))
      combine_rows<T, HD, NT>(a.ws_acc, a.ws_ml, static_cast<T*>(a.out), (size_t)b * a.n_q + (size_t)j * g, g, a.S,
                              reinterpret_cast<float*>(lds + AL.cmb));
  }
}

// ------------------------------------------------------------------ streaming stored-K/V attention (bf16)

// One workgroup of kSaWaves waves per (split s, KV head j, sequence b): the keys
// of blocks sa_first_block(s) .. sa_first_block(s + 1) - 1 of the stored K/V,
// block i to wave i % kSaWaves.  Memory traffic is the K/V rows read once
// (Eq. read_bytes): HBM-bound, so the design keeps loads in flight rather than
// counting flops.  Per block a wave
//  - has the NEXT block's K and V already loading into registers (two
//    register sets, unconditional loads with clamped rows, so the compiler's
//    memory-counter waits stay static);
//  - takes the scores S^T = K q^T on MFMA 16x16x32 bf16: K is the A operand
//    straight from global memory (lane: key lane % 16, 8 dims at 32 c +
//    8 (lane / 16)), q the B operand (lane: query head lane % 16, zero past g),
//    so no cross-lane dot-product reduction is needed;
//  - runs the online softmax in the log2 domain (Eqs. attn_weights /
//    head_output split over keys): the block max over the 4 key lanes of each
//    head by two xor shuffles, p = 2^(s - m), the running sum per lane;
//  - P V on the vector ALUs: V rows are loaded as whole 16-byte chunks (one
//    load instruction covers 64 / (hd / 8) consecutive rows, fully coalesced),
//    each lane keeps fp32 accumulators for 8 columns of each head; the
//    probabilities and the rescale factors pass through a wave-private LDS
//    slot.
// At the end the key groups of each wave are added by xor shuffles, the waves
// merged through LDS (weights 2^(m_w - M), in wave order), and the split's
// state written as a partial in the split-K workspace format, or, with one
// split and out given, normalised straight into out.  The split merge is
// combine_rows, as in every other attention kernel.
template <int HD, int G>
__global__ __launch_bounds__(64 * kSaWaves) __attribute__((amdgpu_waves_per_eu(2))) void stream_attn_kernel(
    AttnArgs a) {
  extern __shared__ __align__(16) char lds[];
  constexpr int NW = kSaWaves, NT = 64 * NW;
  constexpr int NC = HD / 32;    // MFMA K-steps of a score block = V loads per lane per block
  constexpr int CPK = HD / 8;    // 16-byte chunks of a K or V row
  constexpr int KPI = 64 / CPK;  // rows per V load instruction
  static_assert(NC * KPI == kSaBlock, "a block's V rows: NC loads of KPI rows");
  static_assert(G >= 1 && G <= 16, "query heads per KV head");
  constexpr SaLds SL = sa_lds(HD, G);
  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int s = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int g = a.n_q / a.n_kv;
  const int k0 = kSaBlock * sa_first_block(s, a.nblk, a.S);
  const int nk = min(a.T, kSaBlock * sa_first_block(s + 1, a.nblk, a.S)) - k0;  // keys of this split, >= 1
  const int nblk = (nk + kSaBlock - 1) / kSaBlock;
  const int nb = nblk > w ? (nblk - 1 - w) / NW + 1 : 0;  // this wave's blocks: w, w + NW, ...
  const size_t row0 = ((size_t)b * a.n_kv + j) * a.t_cap + a.t_off + k0;
  const uint16_t* Kp = static_cast<const uint16_t*>(a.k) + row0 * HD;
  const uint16_t* Vp = static_cast<const uint16_t*>(a.v) + row0 * HD;
  const int hq = lane & 15;  // query head of this lane's score column

  // q as the MFMA B operand, bf16 as stored
  bf16x8_t qf[NC];
  {
    const uint16_t* qs = static_cast<const uint16_t*>(a.q) + ((size_t)b * a.n_q + (size_t)j * g + min(hq, g - 1)) * HD +
                         8 * (lane >> 4);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      u32x4_t v = *reinterpret_cast<const u32x4_t*>(qs + 32 * c);
      if (hq >= g) v = u32x4_t{0u, 0u, 0u, 0u};
      qf[c] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  // the wave's i-th block (i clamped to its last block) into registers
  auto load = [&](u32x4_t (&kr)[NC], u32x4_t (&vr)[NC], int i) {
    const int kb = kSaBlock * (w + NW * min(i, nb - 1));
    const uint16_t* kp = Kp + (size_t)min(kb + hq, nk - 1) * HD + 8 * (lane >> 4);
#pragma unroll
    for (int c = 0; c < NC; ++c) kr[c] = *reinterpret_cast<const u32x4_t*>(kp + 32 * c);
#pragma unroll
    for (int c = 0; c < NC; ++c)
      vr[c] = *reinterpret_cast<const u32x4_t*>(Vp + (size_t)min(kb + KPI * c + lane / CPK, nk - 1) * HD +
                                                8 * (lane % CPK));
  };

  float m_run = -INFINITY, l_run = 0.0f;
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
  float* Pw = reinterpret_cast<float*>(lds + SL.p) + w * (G + 1) * kSaBlock;  // [G][16] probabilities
  float* Aw = Pw + G * kSaBlock;                                                // [G] rescale factors

  auto attend = [&](const u32x4_t (&kr)[NC], const u32x4_t (&vr)[NC], int i) {
    const int kb = kSaBlock * (w + NW * i);
    f32x4_t sc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int c = 0; c < NC; ++c)
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kr[c]), qf[c], sc, 0, 0, 0);
    // sc[r]: key kb + 4 (lane / 16) + r, query head hq
    float sv[4], bm = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      sv[r] = kb + 4 * (lane >> 4) + r < nk ? sc[r] * ScoreScale<HD>::v : -INFINITY;
      bm = fmaxf(bm, sv[r]);
    }
    bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
    bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
    const float m_new = fmaxf(m_run, bm);  // finite: every attended block holds a key
    const float alpha = exp2f(m_run - m_new);
    float p[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) p[r] = exp2f(sv[r] - m_new);
    l_run = fmaf(l_run, alpha, (p[0] + p[1]) + (p[2] + p[3]));
    m_run = m_new;
    if (hq < G) *reinterpret_cast<float4*>(Pw + hq * kSaBlock + 4 * (lane >> 4)) = make_float4(p[0], p[1], p[2], p[3]);
    if (lane < G) Aw[lane] = alpha;
    __builtin_amdgcn_wave_barrier();  // the wave's LDS writes are ordered before its reads below
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float al = Aw[h];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] *= al;
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int kk = KPI * c + lane / CPK;  // key of this V chunk within the block
      const uint32_t vw[4] = {vr[c].x, vr[c].y, vr[c].z, vr[c].w};
      float v8[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v8[2 * e] = bf_lo(vw[e]);
        v8[2 * e + 1] = bf_hi(vw[e]);
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float pr = Pw[h * kSaBlock + kk];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pr, v8[e], acc[h][e]);
      }
    }
    __builtin_amdgcn_wave_barrier();  // reads of this block's slot before the next block's writes
  };

  // Blocks in pairs, the loop body straight-line (a branch out of its middle
  // made the compiler's register reuse wait for every load in flight).  With
  // an odd count the last pair's second block lies past the split: all its
  // keys are masked, so it leaves the state unchanged (alpha = 1, p = 0).
  // The scheduling barriers keep each refill after the last use of the
  // registers it overwrites: hoisted above it, the refill got fresh registers
  // and a copy back at the loop edge, which waited for every load in flight.
  if (nb > 0) {
    u32x4_t kr0[NC], vr0[NC], kr1[NC], vr1[NC];
    load(kr0, vr0, 0);
    for (int i = 0; i < nb; i += 2) {
      __builtin_amdgcn_sched_barrier(0);
      load(kr1, vr1, i + 1);
      attend(kr0, vr0, i);
      __builtin_amdgcn_sched_barrier(0);
      load(kr0, vr0, i + 2);
      attend(kr1, vr1, i + 1);
    }
  }

  // the wave's state: sums over its key lanes (4 per head for l, KPI per column chunk for acc)
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
#pragma unroll
  for (int o = CPK; o < 64; o <<= 1)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] += __shfl_xor(acc[h][e], o, 64);

  float* ms = reinterpret_cast<float*>(lds + SL.ml);   // [NW][G][2]
  float* as = reinterpret_cast<float*>(lds + SL.acc);  // [NW][G][HD]
  if (lane < G) {
    ms[(w * G + lane) * 2] = m_run;
    ms[(w * G + lane) * 2 + 1] = l_run;
  }
  if (lane < CPK) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float* dst = as + ((size_t)w * G + h) * HD + 8 * lane;
      *reinterpret_cast<float4*>(dst) = make_float4(acc[h][0], acc[h][1], acc[h][2], acc[h][3]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(acc[h][4], acc[h][5], acc[h][6], acc[h][7]);
    }
  }
  __syncthreads();

  // merge of the waves (in wave order): the split's state, or with one split its output
  const bool direct = a.S == 1 && a.out != nullptr;
  for (int i = tid; i < g * HD; i += NT) {
    const int h = i / HD, c = i - h * HD;
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < NW; ++v) M = fmaxf(M, ms[(v * G + h) * 2]);
    float o = 0.0f, L = 0.0f;
#pragma unroll
    for (int v = 0; v < NW; ++v) {
      const float wt = exp2f(ms[(v * G + h) * 2] - M);
      o = fmaf(wt, as[((size_t)v * G + h) * HD + c], o);
      L = fmaf(wt, ms[(v * G + h) * 2 + 1], L);
    }
    const size_t row = (size_t)b * a.n_q + (size_t)j * g + h;
    if (direct) {
      static_cast<uint16_t*>(a.out)[row * HD + c] = from_f<uint16_t>(o / L);
    } else {
      store_dev(a.ws_acc + (row * a.S + s) * HD + c, o);
      if (c == 0) {
        store_dev(a.ws_ml + (row * a.S + s) * 2, M);
        store_dev(a.ws_ml + (row * a.S + s) * 2 + 1, L);
      }
    }
  }
  if (a.out != nullptr && a.S > 1) {
    unsigned long long* ctr = a.ws_done + (size_t)b * a.n_kv + j;
    const unsigned long long before = split_arrive(ctr, 1, reinterpret_cast<unsigned long long*>(lds + SL.ctr));
    if (split_complete(ctr, before, 1, a.S))
      combine_rows<uint16_t, HD, NT, (G <= 2)>(a.ws_acc, a.ws_ml, static_cast<uint16_t*>(a.out),
                                               (size_t)b * a.n_q + (size_t)j * g, g, a.S,
                                               reinterpret_cast<float*>(lds + SL.cmb));
  }
}

// Standalone merge (kvd_combine): one workgroup per (b, query head), the same
// arithmetic as the merge the attention kernels run in their last workgroup.
template <typename T, int HD>
__global__ __launch_bounds__(kNtAttn) void combine_kernel(const float* ws_acc, const float* ws_ml, T* out, int n_q,
                                                          int S) {
  __shared__ float cmb[cmb_floats(kNtAttn, HD)];
  combine_rows<T, HD, kNtAttn>(ws_acc, ws_ml, out, (size_t)blockIdx.y * n_q + blockIdx.x, 1, S, cmb);
}

// ------------------------------------------------------------------ weight packing

// One thread per 16-byte chunk of the packed matrix (see kvd_pack_weights).
// gamma != nullptr: each element becomes bf16(w * gamma[column]) (the exact
// fp32 product, one round-to-nearest-even), kvd_pack_weights_gamma.
__global__ __launch_bounds__(256) void pack_kernel(const uint16_t* w, const uint16_t* gamma, uint16_t* out, int rows,
                                                   int d) {
  const long long chunk = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long n = (long long)rows * d / 8;
  if (chunk >= n) return;
  const int l = (int)(chunk % 64);
  const long long blk = chunk / 64;
  const int kb = (int)(blk % (d / 16));
  const long long rb = blk / (d / 16);
  const int col = 16 * kb + 8 * (l / 32);
  const uint16_t* src = w + (size_t)(rb * 32 + l % 32) * d + col;
  uint4 v = *reinterpret_cast<const uint4*>(src);
  if (gamma != nullptr) {
    const uint4 g = *reinterpret_cast<const uint4*>(gamma + col);
    v.x = pack_bf16x2(bf_lo(v.x) * bf_lo(g.x), bf_hi(v.x) * bf_hi(g.x));
    v.y = pack_bf16x2(bf_lo(v.y) * bf_lo(g.y), bf_hi(v.y) * bf_hi(g.y));
    v.z = pack_bf16x2(bf_lo(v.z) * bf_lo(g.z), bf_hi(v.z) * bf_hi(g.z));
    v.w = pack_bf16x2(bf_lo(v.w) * bf_lo(g.w), bf_hi(v.w) * bf_hi(g.w));
  }
  *reinterpret_cast<uint4*>(out + (size_t)chunk * 8) = v;
}

// ------------------------------------------------------------------ residual checkpoint store

// One workgroup per (16-byte chunk block, row b): dst row b <- src row b.
__global__ __launch_bounds__(256) void copy_rows_kernel(const char* src, size_t src_stride, char* dst, size_t dst_stride,
                                                        int chunks) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= chunks) return;
  const size_t b = blockIdx.y;
  *reinterpret_cast<uint4*>(dst + b * dst_stride + (size_t)c * 16) =
      *reinterpret_cast<const uint4*>(src + b * src_stride + (size_t)c * 16);
}

hipError_t launch_copy_rows(const void* src, size_t src_stride, void* dst, size_t dst_stride, size_t row_bytes, int B,
                            hipStream_t st) {
  const int chunks = (int)(row_bytes / 16);
  hipLaunchKernelGGL(copy_rows_kernel, dim3((unsigned)((chunks + 255) / 256), (unsigned)B), dim3(256), 0, st,
                     static_cast<const char*>(src), src_stride, static_cast<char*>(dst), dst_stride, chunks);
  return hipGetLastError();
}

hipError_t launch_pack(const void* w, const void* gamma, void* out, int rows, int d, hipStream_t st) {
  const long long n = (long long)rows * d / 8;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, static_cast<const uint16_t*>(w),
                     static_cast<const uint16_t*>(gamma), static_cast<uint16_t*>(out), rows, d);
  return hipGetLastError();
}

// ------------------------------------------------------------------ static scratch

// The allocation-free fused call's workspace (split counters, then partials):
// one array per device, held until the process ends.  Host code never names
// the array after set-up: noalloc_scratch() looks up each device's address
// once (with that device current) and every launch, fill and copy takes that
// pointer.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];
}  // namespace

hipError_t noalloc_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

// ------------------------------------------------------------------ launchers

template <typename K>
static hipError_t set_lds(K kernel, size_t bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

// Raise the kernel's dynamic-LDS limit once per process (per kernel and size).
// `done` is the largest size already set; threads that race here may both set
// the attribute, which is idempotent, and the atomic keeps the maximum.
template <typename K>
static hipError_t ensure_lds(K kernel, size_t bytes, std::atomic<size_t>& done) {
  if (bytes <= done.load(std::memory_order_acquire)) return hipSuccess;
  hipError_t e = set_lds(kernel, bytes);
  if (e != hipSuccess) return e;
  size_t cur = done.load(std::memory_order_relaxed);
  while (cur < bytes && !done.compare_exchange_weak(cur, bytes, std::memory_order_release)) {
  }
  return hipSuccess;
}

// Launcher templates take the weight layout L: 0 row-major, 1 packed, 2 packed
// with gamma folded in (kvd_weight_layout).
template <typename T, int HD, int L>
static hipError_t proj_t(const ProjArgs& a, int n_units, hipStream_t st) {
  constexpr int MT = sizeof(T) == 2 ? kMtBf16 : kMtF32;
  const size_t bytes = proj_lds<T>(HD, MT).end + gamma_lds_bytes(a.d);
  static std::atomic<size_t> done{0};
  auto k = proj_kernel<T, HD, MT, L != 0, L == 2>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  const long long ntok = (long long)a.B * a.T;
  const int n_tiles = (int)((ntok + MT - 1) / MT);
  const XcdMap m = xcd_map((long long)n_units * n_tiles);
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(kNtTile), bytes, st, a, m.per, n_tiles, n_units);
  return hipGetLastError();
}

template <int HD, int L>
static hipError_t proj_wide_t(const ProjArgs& a, int n_units, hipStream_t st) {
  const size_t bytes = proj_lds<uint16_t>(HD, kMtWide).end + gamma_lds_bytes(a.d);
  static std::atomic<size_t> done{0};
  auto k = proj_wide_kernel<HD, L != 0, L == 2>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  const int tps = (a.T + kMtWide - 1) / kMtWide;
  const XcdMap m = xcd_map((long long)n_units * a.B * tps);
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(kNtWide), bytes, st, a, m.per, tps, n_units);
  return hipGetLastError();
}

template <int HD, int MT, int NT, int RW, int L>
static hipError_t proj_split_t(const ProjArgs& a, int n_units, hipStream_t st) {
  const size_t bytes = split_lds(RW, MT).end + gamma_lds_bytes(a.d);
  static std::atomic<size_t> done{0};
  auto k = proj_split_kernel<HD, MT, NT, RW, L != 0, L == 2>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  const int tps = (a.T + MT - 1) / MT;
  const XcdMap m = xcd_map(2LL * (HD / RW) * n_units * a.B * tps);
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(NT), bytes, st, a, m.per, tps, n_units);
  return hipGetLastError();
}

template <int HD, int L, int NCH>
static hipError_t stream_t(const ProjArgs& a, hipStream_t st) {
  const int G = stream_group(a.d, a.B * a.T, kLdsPerGroup);
  if (G < 1) return hipErrorInvalidValue;  // validated by the caller
  const size_t bytes = stream_lds(a.d, G).end;
  static std::atomic<size_t> done{0};
  auto k = stream_proj_kernel<HD, L != 0, NCH, L == 2>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  const int qb = a.q_out ? a.n_q * HD / 32 : 0;
  const int kb = a.n_kv_units ? a.n_kv * HD / 32 : 0;
  dim3 grid(qb + 2 * kb, (a.B * a.T + G - 1) / G);
  hipLaunchKernelGGL(k, grid, dim3(64 * kStreamWaves), bytes, st, a, qb, kb, G);
  return hipGetLastError();
}

template <typename T, int HD, int L>
static hipError_t fused_t(const FusedArgs& a, hipStream_t st) {
  constexpr int MT = sizeof(T) == 2 ? kMtBf16 : kMtF32;
  const size_t bytes = fused_lds_bytes<T>(a.n_q / a.n_kv, HD, MT) + gamma_lds_bytes(a.d);
  static std::atomic<size_t> done{0};
  auto k = fused_kernel<T, HD, MT, L != 0, L == 2>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  const int n_tail = fused_tail_tiles<T>(a.n_rec, a.T_tail);
  const int C = n_tail + a.n_rec;
  const XcdMap m = xcd_map((long long)a.n_kv * a.B * C);
  // With stored tail tiles (short items that go first in each head's run) one
  // head per XCD run keeps short items in most runs, so that a grid a little
  // larger than the chip starts its last items on CUs the short ones free.
  const int hg = n_tail > 0 ? 1 : fused_head_group(a.n_kv, HD, m.per);
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(kNtTile), bytes, st, a, m.per, hg);
  return hipGetLastError();
}

template <int HD, int L>
static hipError_t fused_wide_t(const FusedArgs& a, hipStream_t st) {
  const size_t bytes = fused_wide_lds_bytes(a.n_q / a.n_kv, HD) + gamma_lds_bytes(a.d);
  static std::atomic<size_t> done{0};
  auto k = fused_wide_kernel<HD, L != 0, L == 2>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  const int n_tail = fused_tail_tiles<uint16_t>(a.n_rec, a.T_tail);
  const int C = n_tail + a.n_rec;
  const XcdMap m = xcd_map((long long)a.n_kv * a.B * C);
  const int hg = n_tail > 0 ? 1 : fused_head_group(a.n_kv, HD, m.per);
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(kNtWide), bytes, st, a, m.per, hg);
  return hipGetLastError();
}

template <int L>
static hipError_t fused_pair_t(const FusedArgs& a, hipStream_t st) {
  if (a.n_kv % 2 != 0) return hipErrorInvalidValue;
  const size_t bytes = fused_pair_lds_bytes(a.n_q / a.n_kv) + gamma_lds_bytes(a.d);
  static std::atomic<size_t> done{0};
  auto k = fused_pair_kernel<L != 0, L == 2>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  const int n_tail = fused_tail_tiles<uint16_t>(a.n_rec, a.T_tail);
  const int C = n_tail + a.n_rec;
  const int np = a.n_kv / 2;
  const XcdMap m = xcd_map((long long)np * a.B * C);
  // a pair's weight rows are a head_dim 256 head's
  const int hg = n_tail > 0 ? 1 : fused_head_group(np, 256, m.per);
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(kNtWide), bytes, st, a, m.per, hg);
  return hipGetLastError();
}

template <int HD, int MT, int L>
static hipError_t fused_split_t(const FusedArgs& a, hipStream_t st) {
  const size_t bytes = fused_split_lds_bytes(a.n_q / a.n_kv, HD, MT) + gamma_lds_bytes(a.d);
  static std::atomic<size_t> done{0};
  auto k = fused_split_kernel<HD, MT, L != 0, L == 2>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  // items in pairs: an even count per XCD keeps each pair on one XCD
  const long long pairs = (long long)a.n_kv * a.B * a.n_rec;
  const int per = 2 * (int)((pairs + kXcds - 1) / kXcds);
  const int hg = fused_head_group(a.n_kv, HD, per / 2);
  hipLaunchKernelGGL(k, dim3(kXcds * per), dim3(split_nt(HD)), bytes, st, a, per, hg);
  return hipGetLastError();
}

template <typename T, int HD>
static hipError_t attn_t(const AttnArgs& a, hipStream_t st) {
  const size_t bytes = decode_lds_bytes<T>(a.n_q / a.n_kv, HD);
  static std::atomic<size_t> done{0};
  auto k = decode_kernel<T, HD>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, dim3(a.S, a.n_kv, a.B), dim3(kNtAttn), bytes, st, a);
  return hipGetLastError();
}

template <int HD, int G>
static hipError_t stream_attn_t(const AttnArgs& a, hipStream_t st) {
  constexpr size_t bytes = sa_lds(HD, G).end;
  static std::atomic<size_t> done{0};
  auto k = stream_attn_kernel<HD, G>;
  hipError_t e = ensure_lds(k, bytes, done);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, dim3(a.S, a.n_kv, a.B), dim3(64 * kSaWaves), bytes, st, a);
  return hipGetLastError();
}

template <int HD>
static hipError_t stream_attn_g(const AttnArgs& a, hipStream_t st) {
  switch (sa_group(a.n_q / a.n_kv)) {
    case 1: return stream_attn_t<HD, 1>(a, st);
    case 2: return stream_attn_t<HD, 2>(a, st);
    case 3: return stream_attn_t<HD, 3>(a, st);
    case 4: return stream_attn_t<HD, 4>(a, st);
    case 6: return stream_attn_t<HD, 6>(a, st);
    case 8: return stream_attn_t<HD, 8>(a, st);
    case 16: return stream_attn_t<HD, 16>(a, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int HD>
static hipError_t combine_t(const float* ws_acc, const float* ws_ml, void* out, int n_q, int B, int S,
                            hipStream_t st) {
  hipLaunchKernelGGL((combine_kernel<T, HD>), dim3(n_q, B), dim3(kNtAttn), 0, st, ws_acc, ws_ml,
                     static_cast<T*>(out), n_q, S);
  return hipGetLastError();
}

#define KVD_DISPATCH(DT, HDV, CALL_BF16, CALL_F32)         \
  switch (HDV) {                                           \
    case 64:                                               \
      return DT ? CALL_BF16(64) : CALL_F32(64);            \
    case 128:                                              \
      return DT ? CALL_BF16(128) : CALL_F32(128);          \
    case 256:                                              \
      return DT ? CALL_BF16(256) : CALL_F32(256);          \
    default:                                               \
      return hipErrorInvalidValue;                         \
  }

// f(IC<L>{}) for layout L in 0..2
template <class F>
static hipError_t with_layout(int layout, const F& f) {
  switch (layout) {
    case 0: return f(IC<0>{});
    case 1: return f(IC<1>{});
    case 2: return f(IC<2>{});
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_proj(const ProjArgs& a, int dtype_bf16, int hd, int layout, int n_units, hipStream_t st) {
  if (dtype_bf16 && (hd == 128 || hd == 256) &&
      narrow_prefill(2LL * (hd / kRwNarrow) * n_units * a.B * ((a.T + kMtNarrow - 1) / kMtNarrow))) {
    return with_layout(layout, [&](auto lc) -> hipError_t {
      constexpr int L = decltype(lc)::value;
      return hd == 256 ? proj_split_t<256, kMtNarrow, kNtNarrow, kRwNarrow, L>(a, n_units, st)
                       : proj_split_t<128, kMtNarrow, kNtNarrow, kRwNarrow, L>(a, n_units, st);
    });
  }
  if (dtype_bf16 && (hd == 128 || hd == 256) &&
      wide_prefill((long long)n_units * a.B * ((a.T + kMtWide - 1) / kMtWide)) &&
      proj_lds<uint16_t>(hd, kMtWide).end + gamma_lds_bytes(a.d) <= kLdsPerGroup) {
    return with_layout(layout, [&](auto lc) -> hipError_t {
      constexpr int L = decltype(lc)::value;
      return hd == 256 ? proj_wide_t<256, L>(a, n_units, st) : proj_wide_t<128, L>(a, n_units, st);
    });
  }
  if (dtype_bf16 && split_prefill(hd, a.T, 2LL * n_units * a.B * ((a.T + kMtSplit - 1) / kMtSplit))) {
    return with_layout(layout, [&](auto lc) -> hipError_t {
      constexpr int L = decltype(lc)::value;
      return hd == 256 ? proj_split_t<256, kMtSplit, split_nt(256), 256, L>(a, n_units, st)
                       : proj_split_t<128, kMtSplit, split_nt(128), 128, L>(a, n_units, st);
    });
  }
#define PB(H) with_layout(layout, [&](auto lc) { return proj_t<uint16_t, H, decltype(lc)::value>(a, n_units, st); })
#define PF(H) proj_t<float, H, 0>(a, n_units, st)
  KVD_DISPATCH(dtype_bf16, hd, PB, PF)
#undef PB
#undef PF
}

// d = 2560 (Gemma-3-4B) and 1536 (Qwen2.5-1.5B) get a compile-time chunk count.
template <int HD, int L>
static hipError_t stream_nch(const ProjArgs& a, hipStream_t st) {
  switch (a.d / (kKT * kStreamChunk)) {
    case 20: if (a.d == 20 * kKT * kStreamChunk) return stream_t<HD, L, 20>(a, st); break;
    case 12: if (a.d == 12 * kKT * kStreamChunk) return stream_t<HD, L, 12>(a, st); break;
    default: break;
  }
  return stream_t<HD, L, 0>(a, st);
}

hipError_t launch_project_current(const ProjArgs& a, int dtype_bf16, int hd, int layout, int n_units,
                                  hipStream_t st) {
  if (!dtype_bf16) return launch_proj(a, 0, hd, 0, n_units, st);
  return with_layout(layout, [&](auto lc) -> hipError_t {
    constexpr int L = decltype(lc)::value;
    switch (hd) {
      case 64: return stream_nch<64, L>(a, st);
      case 128: return stream_nch<128, L>(a, st);
      case 256: return stream_nch<256, L>(a, st);
      default: return hipErrorInvalidValue;
    }
  });
}

hipError_t launch_fused(const FusedArgs& a, int dtype_bf16, int hd, int layout, int engine, hipStream_t st) {
  if (engine == kFusedSplit || engine == kFusedSplit64) {
    if (!dtype_bf16) return hipErrorInvalidValue;
    const bool m64 = engine == kFusedSplit64;
    return with_layout(layout, [&](auto lc) -> hipError_t {
      constexpr int L = decltype(lc)::value;
      switch (hd) {
        case 128: return m64 ? fused_split_t<128, 64, L>(a, st) : fused_split_t<128, kMtSplit, L>(a, st);
        case 256: return m64 ? fused_split_t<256, 64, L>(a, st) : fused_split_t<256, kMtSplit, L>(a, st);
        default: return hipErrorInvalidValue;
      }
    });
  }
  if (engine == kFusedPair) {
    if (!dtype_bf16 || hd != 128) return hipErrorInvalidValue;
    return with_layout(layout, [&](auto lc) -> hipError_t { return fused_pair_t<decltype(lc)::value>(a, st); });
  }
  if (engine == kFusedWide) {
    if (!dtype_bf16) return hipErrorInvalidValue;
    return with_layout(layout, [&](auto lc) -> hipError_t {
      constexpr int L = decltype(lc)::value;
      switch (hd) {
        case 128: return fused_wide_t<128, L>(a, st);
        case 256: return fused_wide_t<256, L>(a, st);
        default: return hipErrorInvalidValue;
      }
    });
  }
  hipError_t e;
#define FB(H) with_layout(layout, [&](auto lc) { return fused_t<uint16_t, H, decltype(lc)::value>(a, st); })
#define FF(H) fused_t<float, H, 0>(a, st)
  e = [&]() -> hipError_t { KVD_DISPATCH(dtype_bf16, hd, FB, FF) }();
#undef FB
#undef FF
  return e;
}

hipError_t launch_combine(const float* ws_acc, const float* ws_ml, void* out, int n_q, int B, int S, int dtype_bf16,
                          int hd, hipStream_t st) {
#define CB(H) combine_t<uint16_t, H>(ws_acc, ws_ml, out, n_q, B, S, st)
#define CF(H) combine_t<float, H>(ws_acc, ws_ml, out, n_q, B, S, st)
  KVD_DISPATCH(dtype_bf16, hd, CB, CF)
#undef CB
#undef CF
}

hipError_t launch_decode(const AttnArgs& a, int dtype_bf16, int hd, hipStream_t st) {
#define AB(H) stream_attn_g<H>(a, st)
#define AF(H) attn_t<float, H>(a, st)
  KVD_DISPATCH(dtype_bf16, hd, AB, AF)
#undef AB
#undef AF
}

}  // namespace kvd
