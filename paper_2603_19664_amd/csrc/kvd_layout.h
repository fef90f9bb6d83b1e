// Launch geometry and LDS carve-up shared by the host launchers and the
// kernels of libkvd.  Plain constexpr arithmetic, usable on host and device.
#pragma once
#include <stddef.h>
#include <stdint.h>

namespace kvd {

constexpr int kNtTile = 512;    // threads of the recompute / fused kernels (8 wave64 waves)
constexpr int kNtAttn = 512;    // threads of the stored-K/V attention and combine kernels
constexpr int kKT = 64;         // d-elements per K-step of the projection GEMM
constexpr int kTile = 64;       // keys per attention tile (one split-K partial)
constexpr int kMaxGroup = 16;   // max query heads per KV head
constexpr int kMaxPairs = 128;  // head_dim / 2 for head_dim <= 256
constexpr int kXcds = 8;        // MI355X: workgroups are dispatched round-robin over 8 XCDs
constexpr int kDepth = 4;       // K-steps of weights / residuals in flight in the recompute GEMM

// Tokens per workgroup of the recompute engines.
constexpr int kMtBf16 = 64;
constexpr int kMtF32 = 64;

// The wide bf16 engine of the fused kernel (head_dim 128 / 256): 128 tokens per
// workgroup on 8 waves, two per SIMD.  Used when the call has at least
// kWideMinTiles such tiles (one per CU: a full round), so that the larger tile
// does not leave CUs idle.
constexpr int kNtWide = 512;
constexpr int kMtWide = 128;
constexpr int kWideMinTiles = 256;

// The split engine (bf16, head_dim 128 / 256): a 128-token tile of one half
// (a KV head's K rows, or its V rows) per workgroup of 4 waves, one per SIMD.
// The K and V halves of a tile run as two workgroups, so a grid has as many
// workgroups as with 64-token tiles of both halves while each CU streams half
// the weight bytes per flop.  The K/V tile in LDS holds one half: row stride
// split_ld(hd) elements.
constexpr int kMtSplit = 128;
// head_dim 256: 8 waves of one 32-row block each (two per SIMD); head_dim 128:
// 4 waves (the half has 128 rows).
constexpr int split_nt(int hd) { return hd == 256 ? 512 : 256; }
// The fused call on the split engine: the V role of chunk c waits for bit c of
// its (sequence, KV head)'s completion words, which the K role sets once its
// probabilities are out; the words are cleared by the workgroup that merges
// the splits.  At most 64 * kSplitBitWords chunks per sequence.
constexpr int kSplitBitWords = 4;
constexpr int kSplitMaxChunks = 64 * kSplitBitWords;
// Polls of the V role's bounded wait (about 0.1 s); past it the chunk's partial
// is written as NaN, so the call's output shows the failure.
constexpr unsigned kSplitSpinLimit = 1u << 17;
// Floats of one chunk's exchange record for group size g and mt-token chunks
// (rows: mt plus a folded tail of up to 4, fold_rows).
constexpr int split_xf(int g, int mt) { return (g * (mt + 4) + 2 * g + 3) / 4 * 4; }
// The fused call takes 64-token chunks on the split engine when its 64-token
// grid of both halves (n_kv * B * ceil(T_rec / 64) workgroups) would fill at most
// this many CUs (half the chip): sliding-window layers and short contexts at
// small batch, where each workgroup's K-loop over d_model sets the time.
constexpr long long kSplit64MaxTiles = 128;
constexpr int split_ld(int hd) { return hd + 8; }
// Prefill / recompute (kvd_recompute_kv, the block forward's projections) runs
// on the split engine for bf16 at head_dim 256, and at head_dim 128 when its
// grid (wgs workgroups) fills at least two rounds of the chip: measured on
// MI355X against 64-token tiles of both halves, 8-15% faster at head_dim 256
// (Gemma-3-4B shape, 512..8192 tokens); at head_dim 128 the 4-wave layout is
// 8-10% faster on 512-workgroup grids and 27% slower on 64 (Qwen2.5-1.5B shape).
// Its tiles hold the tokens of one sequence, so sequences shorter than half a
// tile stay on 64-token tiles.
constexpr bool split_prefill(int hd, int T, long long wgs) {
  return T >= kMtSplit / 2 && (hd == 256 || (hd == 128 && wgs >= 512));
}
// The narrow tile of the split engine: 128 rows of one half for 64 tokens, 4
// waves of one 32-row block each, for prefill / recompute calls whose grid of
// narrow tiles (wgs workgroups) holds at most kNarrowMaxWgs: calls too small to
// fill the chip with larger tiles (the evicted-token recomputes of a decode
// step), where each workgroup's K-loop over d_model, not the work, sets the time.
constexpr int kMtNarrow = 64;
constexpr int kNtNarrow = 256;
constexpr int kRwNarrow = 128;
constexpr long long kNarrowMaxWgs = 512;
constexpr bool narrow_prefill(long long wgs) { return wgs <= kNarrowMaxWgs; }
// Prefill on WideTile's 128-token tiles of both halves: calls with at least a
// full round of them (kWideMinTiles; each weight fragment then feeds four MFMAs
// instead of the split engine's two), where their LDS fits.
constexpr bool wide_prefill(long long wgs) { return wgs >= kWideMinTiles; }

// A stored tail of at most fold_rows<T>() rows (a decode step's current token)
// joins the split of the last recomputed tile of a fused call: the rows are
// copied into LDS while that tile is recomputed and attended with its keys.
// Longer tails get one split per 64-row tile.  bf16 only: the fp32 engine's
// K/V tile leaves no LDS for the extra rows at head_dim 256.
template <typename T>
constexpr int fold_rows() { return sizeof(T) == 2 ? 4 : 0; }
template <typename T>
constexpr bool fold_tail(int n_rec, int T_tail) { return n_rec > 0 && T_tail > 0 && T_tail <= fold_rows<T>(); }
// Splits of a stored-K/V attention call over Tk keys: one per 64-key tile, and
// a remainder of at most fold_rows<T>() keys joins the tile before it (so that a
// context that is a multiple of 64 plus the current token fills its grid
// exactly and is chunked as the fused kernel chunks it).
template <typename T>
constexpr int decode_splits(int Tk) {
  const int r = Tk % kTile;
  return Tk > kTile && r > 0 && r <= fold_rows<T>() ? Tk / kTile : (Tk + kTile - 1) / kTile;
}
// Keys per lane of the attention tiles (up to 64 + fold_rows<T>() keys).
template <typename T>
constexpr int tile_kpl() { return kTile + fold_rows<T>() > 64 ? 2 : 1; }
// Splits of a fused call: one per recomputed tile, plus the stored tail's tiles
// unless the tail is folded: one per 64 rows, a remainder of at most
// fold_rows<T>() rows joining the tile before it (as decode_splits chunks
// stored keys), so that a stored window plus the current token adds no
// workgroup for that one row.
template <typename T>
constexpr int fused_tail_tiles(int n_rec, int T_tail) {
  return fold_tail<T>(n_rec, T_tail) ? 0 : decode_splits<T>(T_tail);
}

// Streaming projection (current-token q/K/V): tokens per workgroup.
constexpr int kProjTok = 16;

constexpr size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
constexpr size_t kLdsPerGroup = 160 * 1024;  // LDS a workgroup may use on gfx950

// Row strides (elements) of the LDS tiles; the +8 / +4 padding keeps the
// 16-byte row reads of a wave on distinct LDS banks.
template <typename T> struct Pad;
template <> struct Pad<uint16_t> { static constexpr int kv = 8; static constexpr int h = 8; };
template <> struct Pad<float> { static constexpr int kv = 4; static constexpr int h = 4; };

template <typename T>
constexpr int kv_ld(int hd) { return 2 * hd + Pad<T>::kv; }
template <typename T>
constexpr int h_ld(void) { return kKT + Pad<T>::h; }

// LDS layout of the attention part (decode / fused kernels); g = group size.
struct AttnLds {
  size_t q, s, red, ml, cmb, ctr, end;
};
// Split merge (combine_rows): blocks of 64 splits; the (max, sum) pairs of the
// first kCmbKeep blocks stay in registers.  LDS floats: rows-per-pass (up to
// two per nt / hd threads) x (64 weights + max and sum).
constexpr int kCmbKeep = 2;
constexpr size_t cmb_floats(int nt, int hd) { return (size_t)(2 * (nt / hd)) * 66; }
// Key splits of the P V phase of a tile's attention: fixed by the group size
// alone, so that kernels with different thread counts add in the same order.
constexpr int attn_ts(int g) { return g >= 8 ? 1 : 8 / g; }
// Scratch of a tile's attention: the scores of up to 64 keys per (head, 64-dim
// part) per pass over `rows`, then the P V partial sums of the key splits.
constexpr size_t red_floats(int g, int hd, int rows) {
  const size_t sc = (size_t)((rows + 63) / 64) * g * hd;
  const size_t pv = (size_t)attn_ts(g) * g * hd;
  return sc > pv ? sc : pv;
}
// q, probabilities, the scratch `red` (scores, then the key splits' P V
// partial sums, which write_partial adds as it writes the tile's output), (max,
// sum), the split counter's broadcast.  The split merge, which runs after all
// tiles, reuses `red` as well.
__attribute__((always_inline)) constexpr AttnLds attn_lds(size_t base, int g, int hd, int rows) {
  AttnLds L{};
  L.q = align_up(base, 16);
  L.s = align_up(L.q + sizeof(float) * g * hd, 16);
  L.red = align_up(L.s + sizeof(float) * g * rows, 16);
  const size_t rf = red_floats(g, hd, rows), cf = cmb_floats(512, hd);
  L.cmb = L.red;
  L.ml = align_up(L.red + sizeof(float) * (rf > cf ? rf : cf), 16);
  L.ctr = align_up(L.ml + sizeof(float) * 2 * g, 16);  // split counter broadcast
  L.end = align_up(L.ctr + sizeof(unsigned long long), 16);
  return L;
}

// LDS layout of the recompute engine: staged h-bar tiles, the K/V tile (aliases
// the staging buffers), per-token 1/rms and positions, and the RoPE frequency
// table.  bf16: a ring of kDepth K-steps of mt tokens x kKT in MFMA B-fragment
// order; fp32: one [mt][h_ld] tile.
struct ProjLds {
  size_t hst, kv, rinv, pos, rev, end;
};
// `extra` rows after the tile's mt are filled during the K-loop (a folded tail),
// so the tile is placed to keep them clear of the staging buffers.
template <typename T>
constexpr ProjLds proj_lds(int hd, int mt, int extra = 0) {
  ProjLds L{};
  L.rev = 0;                                                       // double[kMaxPairs]
  L.rinv = align_up(L.rev + sizeof(double) * kMaxPairs, 16);        // float[mt]
  L.pos = align_up(L.rinv + sizeof(float) * mt, 16);                // int[mt]
  L.hst = align_up(L.pos + sizeof(int) * mt, 16);
  size_t hst_end = L.hst + (sizeof(T) == 2 ? sizeof(T) * kDepth * mt * kKT : sizeof(T) * 2 * mt * h_ld<T>());
  const size_t row = sizeof(T) * kv_ld<T>(hd);
  L.kv = extra > 0 && L.hst + mt * row < hst_end ? hst_end - mt * row : L.hst;  // T[mt + extra][kv_ld]
  size_t kv_end = L.kv + row * (mt + extra);
  L.end = align_up(hst_end > kv_end ? hst_end : kv_end, 16);
  return L;
}

// The split engine's LDS: RoPE table, 1/rms and positions, the staging ring of
// kDepth K-steps of mt tokens, and the one-half K/V tile [mt + extra][split_ld]
// placed (as in proj_lds) so that its rows mt .. (filled during the K-loop)
// stay clear of the ring.
constexpr ProjLds split_lds(int hd, int mt, int extra = 0) {
  ProjLds L{};
  L.rev = 0;
  L.rinv = align_up(L.rev + sizeof(double) * kMaxPairs, 16);
  L.pos = align_up(L.rinv + sizeof(float) * mt, 16);
  L.hst = align_up(L.pos + sizeof(int) * mt, 16);
  const size_t hst_end = L.hst + sizeof(uint16_t) * kDepth * mt * kKT;
  const size_t row = sizeof(uint16_t) * split_ld(hd);
  L.kv = extra > 0 && L.hst + mt * row < hst_end ? hst_end - mt * row : L.hst;
  const size_t kv_end = L.kv + row * (mt + extra);
  L.end = align_up(hst_end > kv_end ? hst_end : kv_end, 16);
  return L;
}

// gamma (bf16, [d]) of the bf16 recompute engine sits after a kernel's other LDS.
constexpr size_t gamma_lds_bytes(int d) { return align_up((size_t)2 * d, 16); }

template <typename T>
constexpr size_t decode_lds_bytes(int g, int hd) {
  // K/V tile (with room for a folded remainder) followed by the attention scratch.
  return attn_lds(align_up(sizeof(T) * (kTile + fold_rows<T>()) * kv_ld<T>(hd), 16), g, hd, kTile + fold_rows<T>()).end;
}

template <typename T>
constexpr size_t fused_lds_bytes(int g, int hd, int mt) {
  return attn_lds(proj_lds<T>(hd, mt, fold_rows<T>()).end, g, hd, mt + fold_rows<T>()).end;
}
// The fused kernel on the split engine: a folded tail of up to fold rows.
constexpr size_t fused_split_lds_bytes(int g, int hd, int mt) {
  return attn_lds(split_lds(hd, mt, 4).end, g, hd, mt + 4).end;
}
// The wide fused kernel: 128-key tiles plus a folded tail.
constexpr size_t fused_wide_lds_bytes(int g, int hd) {
  return attn_lds(proj_lds<uint16_t>(hd, kMtWide, fold_rows<uint16_t>()).end, g, hd, kMtWide + fold_rows<uint16_t>())
      .end;
}
// The pair fused kernel (head_dim 128, two KV heads per 128-token tile): the
// head_dim 256 wide tile's LDS, whose K|V rows hold both heads, then one head
// group's attention scratch; its q region (g x 128 floats) holds both groups'
// raw bf16 q rows.
constexpr size_t fused_pair_lds_bytes(int g) {
  return attn_lds(proj_lds<uint16_t>(256, kMtWide, fold_rows<uint16_t>()).end, g, 128,
                  kMtWide + fold_rows<uint16_t>())
      .end;
}

// Streaming projection (current-token q/K/V): one workgroup of kStreamWaves
// waves per 32 weight rows.  Waves 1.. keep kStreamDepth chunks of the rows'
// MFMA A fragments in flight in registers and write each chunk (kStreamChunk
// K-steps: 32 rows x 64 x bf16 = 4 KiB per K-step) into an LDS ring of
// kStreamSlots slots one chunk ahead of its use; wave 0 runs the MFMA chain.
// LDS: RoPE table, 1/rms and positions of up to kProjTok tokens, gamma, the ring,
// then the raw residual rows of the workgroup's token group (G rows, for the sums
// of squares) and the same rows scaled by gamma (the MFMA B operand).
constexpr int kStreamWaves = 5;
constexpr int kStreamChunk = 2;
constexpr int kStreamSlots = 4;
// Chunks in flight per loader: 6 (48 KiB of weights per workgroup).  A deeper
// ring requests more of the weights at once at the start, and the chain's
// first chunks then wait behind them (measured on the decode step's current
// token, Gemma-3-4B layer: 8.58 us per call at 10 chunks, 8.06 at 6, 8.22 at 4).
constexpr int kStreamDepth = 6;
// A bf16 recompute runs on the streaming projection (its MFMA chain is the tile
// engine's, so the K/V are identical) while that kernel's grid, one workgroup
// per (32 K/V rows, group of up to kProjTok tokens), has at most this many
// workgroups: about two rounds of the chip.  The tile engine takes one whole
// K-loop over d_model per 64-token tile whatever the count (55 us at d 2560,
// 25 us at d 1536, measured); the streaming kernel's time grows with its rounds
// and wins up to two of them (Gemma-3-4B shape: 128 tokens in 36 us; Qwen2.5-
// 1.5B shape: 512 tokens in 21 us).
constexpr long long kStreamRecomputeMaxWgs = 512;
// head_dim 256: against the split engine's narrow tiles (about 35 us for any
// recompute of up to ~1000 tokens at d 2560, measured) the streaming kernel
// wins up to ~100 tokens (its token groups are 11 rows there, LDS-bound: 64
// tokens are 384 workgroups, 24 us; 128 tokens 768 workgroups, 35 us).
constexpr long long kStreamRecomputeMaxWgsHd256 = 640;
constexpr size_t kStreamSlotBytes = (size_t)32 * kKT * 2 * kStreamChunk;
struct StreamLds {
  size_t rev, rinv, pos, gam, ring, hb, hs, end;
};
constexpr int stream_h_ld(int d) { return d + 8; }
constexpr StreamLds stream_lds(int d, int G) {
  StreamLds L{};
  L.rev = 0;
  L.rinv = align_up(L.rev + sizeof(double) * kMaxPairs, 16);
  L.pos = align_up(L.rinv + sizeof(float) * kProjTok, 16);
  L.gam = align_up(L.pos + sizeof(int) * kProjTok, 16);
  L.ring = align_up(L.gam + sizeof(uint16_t) * d, 16);
  L.hb = L.ring + kStreamSlotBytes * kStreamSlots;
  L.hs = align_up(L.hb + sizeof(uint16_t) * G * stream_h_ld(d), 16);
  L.end = align_up(L.hs + sizeof(uint16_t) * G * stream_h_ld(d), 16);
  return L;
}
// Tokens per workgroup of the streaming projection: up to kProjTok, as many as
// the LDS left after the ring holds (0: not even one row fits).
constexpr int stream_group(int d, int B, size_t lds_limit) {
  int G = B < kProjTok ? B : kProjTok;
  while (G > 0 && stream_lds(d, G).end > lds_limit) --G;
  return G;
}

// Streaming stored-K/V attention (bf16 kvd_decode_attn / kvd_cached_attn):
// kSaWaves waves per workgroup, one workgroup per (key split, KV head,
// sequence).  A split's keys go in blocks of kSaBlock (one 16-key MFMA score
// block), block i to wave i % kSaWaves; each wave keeps the next block's K/V
// loads in flight while it attends the current one.
constexpr int kSaWaves = 4;
constexpr int kSaBlock = 16;
// Workgroups the split policy aims for by default: one per CU.  Measured on
// MI355X (Gemma-3-4B layer, B = 1..64): a larger target adds splits whose merge
// (one remote round trip per block of 64, after an arrival per split) costs
// more than the extra parallelism gains.
constexpr int kSaTargetWgs = 256;
// Query heads per KV head the kernel is compiled for: the smallest of 1, 2, 3,
// 4, 6, 8, 16 that is >= g (heads g .. G-1 are computed on zero queries and
// never stored).
constexpr int sa_group(int g) { return g <= 4 ? g : g <= 6 ? 6 : g <= 8 ? 8 : 16; }
// Split count S for T keys and `pairs` = B * n_kv (sequence, KV head) pairs:
// about `target` workgroups in all, at most kSaMaxSplits and at most one split
// per 16-key block.  Split s
// takes blocks sa_first_block(s) .. sa_first_block(s + 1) - 1 of the nblk, so the
// splits' block counts differ by at most one, every split holds at least one
// key, and S never decreases as T grows (a workspace sized for the longest call
// serves the shorter ones).
struct SaSplit {
  int nblk, S;
};
// At most kSaMaxSplits splits: each split adds an arrival on its (sequence, KV
// head) counter and a partial to merge, and past 32 that cost more than the
// parallelism gained (measured, Gemma-3-4B layer, B = 1: 4097 keys in 15.2 us
// with 32 splits, 19.3 us with 64, 25.1 us with 128).
constexpr int kSaMaxSplits = 32;
constexpr SaSplit sa_split(long long pairs, int T, int target) {
  SaSplit r{};
  r.nblk = (T + kSaBlock - 1) / kSaBlock;
  long long s = pairs > 0 ? (target + pairs - 1) / pairs : 1;
  if (s < 1) s = 1;
  if (s > kSaMaxSplits) s = kSaMaxSplits;
  if (s > r.nblk) s = r.nblk;
  r.S = (int)s;
  return r;
}
constexpr int sa_first_block(int s, int nblk, int S) {
  return (int)((long long)s * nblk / S);
}
// LDS of the streaming kernel: per wave the block's probabilities [G][16] and
// rescale factors [16]; the waves' states [kSaWaves][G][hd] and (max, sum)
// [kSaWaves][G][2] for the workgroup merge; the split merge (combine_rows)
// reuses the state area; the split counter's broadcast.
struct SaLds {
  size_t p, acc, ml, cmb, ctr, end;
};
constexpr SaLds sa_lds(int hd, int G) {
  SaLds L{};
  L.p = 0;
  L.acc = align_up(L.p + sizeof(float) * kSaWaves * (G + 1) * kSaBlock, 16);
  L.ml = align_up(L.acc + sizeof(float) * kSaWaves * G * hd, 16);
  const size_t merge_end = align_up(L.ml + sizeof(float) * kSaWaves * G * 2, 16);
  L.cmb = L.acc;
  const size_t cmb_end = L.cmb + sizeof(float) * cmb_floats(64 * kSaWaves, hd);
  L.ctr = align_up(merge_end > cmb_end ? merge_end : cmb_end, 16);
  L.end = align_up(L.ctr + sizeof(unsigned long long), 16);
  return L;
}

// Bytes of the static per-device scratch of kvd_fused_recompute_attn_noalloc:
// enough for the split-K workspace of every measured workload (the largest,
// a Gemma-3-4B layer at B = 64 and 2048 context tokens, needs ~17 MB).
constexpr size_t kNoAllocScratchBytes = (size_t)32 << 20;

// Workgroup -> work item remap that keeps the items of one XCD contiguous:
// hardware dispatch sends workgroup w to XCD w % 8, so XCD x runs items
// x*per .. x*per+per-1, and units that share weights land on the same L2.
struct XcdMap {
  int per;    // items per XCD
  int grid;   // workgroups to launch (kXcds * per)
};
constexpr XcdMap xcd_map(long long n_items) {
  XcdMap m{};
  m.per = (int)((n_items + kXcds - 1) / kXcds);
  m.grid = kXcds * m.per;
  return m;
}

// Heads per group in the fused kernel's item order: per XCD, per items are hg
// heads x per / hg chunks, and the XCD's L2 takes (per / hg) residual tiles of
// 64 d-vectors plus hg heads' W_k | W_v (2 hd d-vectors each).  Their sum is
// least at hg^2 = 32 per / hd; the largest power of two at or below that which
// divides n_kv.
constexpr int fused_head_group(int n_kv, int hd, int per) {
  int hg = 1;
  while (n_kv % (2 * hg) == 0 && (long long)(2 * hg) * (2 * hg) * hd <= 32LL * per) hg *= 2;
  return hg;
}

}  // namespace kvd
