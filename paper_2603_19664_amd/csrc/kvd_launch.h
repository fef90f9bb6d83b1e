// Kernel argument blocks and launcher entry points shared by the C ABI layer
// (kvd_api.cpp) and the kernels (kvd_kernels.hip).  Internal to libkvd.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvd_layout.h"

namespace kvd {

// RMSNorm + projection + RoPE of B*T token rows.  grid.y enumerates units:
// y < n_kv_units -> KV head y (its K rows get RoPE, V rows do not, written to
// k_out / v_out); otherwise query heads 2u, 2u+1 (u = y - n_kv_units), written to
// q_out [B][n_q][HD] (T must then be 1).
struct ProjArgs {
  const void* h;
  const void* gamma;
  const void* w_k;
  const void* w_v;
  const void* w_q;
  const int32_t* pos0;
  void* k_out;
  void* v_out;
  void* q_out;  // [B][T][n_q][hd] (q units)
  long long h_ld;
  int kv_t_cap, kv_t_off;
  int d, n_q, n_kv, B, T, n_kv_units;
  float eps;
  double rev[kMaxPairs];  // RoPE frequency of pair i in revolutions per position
};

// Fused recompute + attention.  grid = (S, n_kv, B) with S = n_rec + n_tail
// chunks of the tile size; chunk s < n_rec recomputes residual rows
// s*MT .. s*MT+MT-1, the rest attend stored tail rows.
struct FusedArgs {
  const void* q;
  const void* h;
  long long h_ld;
  const void* gamma;
  const void* w_k;
  const void* w_v;
  const int32_t* pos0;  // [B] position of residual row 0; nullptr: 0 for every sequence
  const void* tk;
  const void* tv;
  int tail_t_cap, tail_t_off, T_tail;
  void* dbg_k;
  void* dbg_v;
  int dbg_t_cap, dbg_t_off;
  float* ws_acc;
  float* ws_ml;
  unsigned long long* ws_done;  // [B][n_kv] split counters (zero between calls)
  void* out;
  int d, n_q, n_kv, B, T_rec, n_rec, S;
  float eps;
  // split engine: per (b, KV head) kSplitBitWords words of K-role completion
  // bits (zero between calls), and per (b, KV head, chunk) xf floats of the
  // K role's probabilities [g][kMtSplit + fold rows] and (max, sum) [g][2]
  unsigned long long* ws_bits;
  float* xch;
  int xf;
  double rev[kMaxPairs];
};

// Split-K attention over stored K/V.  fp32: S = decode_splits(T) chunks of
// kTile keys (decode_kernel).  bf16: S splits of the nblk 16-key blocks
// (sa_first_block), one streaming workgroup each (stream_attn_kernel).  out == nullptr:
// partials only; otherwise the workgroup that completes the splits of (b, KV
// head) merges them into out (with S == 1 the one workgroup writes out
// directly).  The same holds for FusedArgs::out.
struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  int t_cap, t_off;
  void* out;
  float* ws_acc;
  float* ws_ml;
  unsigned long long* ws_done;
  int B, T, n_q, n_kv, S;
  int nblk;  // bf16: 16-key blocks of the T keys
};

// Block-forward projection on the tile engine (bf16): out = epilogue(x W^T) for
// the M = B * T token rows of x [M][K], 512 output features per workgroup.
//   kEpiResidual: out[m][n] = res[m][n] + (x W^T)[m][n], W [N][K] (N % 512 == 0);
//   kEpiSwiglu:   out[m][f] = SiLU(g) * u with g = (xbar W^T)[m][f], u = (xbar W2^T)[m][f],
//                 W, W2 [N][K] (N % 256 == 0), xbar = RMSNorm(x; gamma).
// norm: the activation rows are RMS-normalised with gamma (1/rms on the
// accumulators, gamma on the staged operand); otherwise gamma is a vector of ones.
enum { kEpiResidual = 0, kEpiSwiglu = 1 };
struct GemmArgs {
  const void* x;
  const void* gamma;
  const void* w;
  const void* w2;
  const void* res;
  void* out;
  int M, K, N;
  int norm;
  float eps;
};
hipError_t launch_gemm(const GemmArgs& a, int epi, int packed, hipStream_t st);

// Causal prefill attention (bf16): out[b][t][h*hd .. h*hd+hd-1] = sum over keys
// j <= t of softmax_j(q[b][t][h] . K[b][h/g][j] / sqrt(hd)) V[b][h/g][j].
//   q [B][T][n_q][hd]; K, V [B][n_kv][T][hd]; out [B][T][n_q * hd].
// Query block qb (rows 128 qb ..) attends nkb = last row / 64 + 1 key blocks of
// 64.  When the blocks are too few and too unequal to fill the chip, a block's
// key range is split into np = ceil(nkb / P) parts of near-equal length, one
// workgroup each; the parts' states (unnormalised O, running max and sum) meet in
// `part`, and the last part to arrive (counter in `ctr`, zero before the launch)
// merges them in part order.  P and NP (the most parts of any block) come from
// prefill_split; with NP == 1 nothing is split and part / ctr are unused.
constexpr int kPrefillOrderMax = 256;
struct PrefillSplit {
  int P, NP;
  int n_order;  // entries of order (0: too many; rank r is then query block nqb - 1 - r, part 0, unsplit)
  unsigned order[kPrefillOrderMax];  // (qb << 8) | part, longest part first
};
struct PrefillArgs {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  int B, T, n_q, n_kv;
  int P, NP;
  float* part;               // [B][n_q][nqb][NP][prefill_part_floats(hd)]
  unsigned long long* ctr;   // [B][n_q][nqb]
  int n_order;
  unsigned order[kPrefillOrderMax];
};
PrefillSplit prefill_split(int B, int T, int n_q);
size_t prefill_part_floats(int hd);
hipError_t launch_prefill_attn(const PrefillArgs& a, int hd, hipStream_t st);

// dst[i] = 1.0 (bf16) for i < n.
hipError_t launch_fill_ones_bf16(void* dst, int n, hipStream_t st);
// dst[i] = 0 (64-bit words) for i < n.
hipError_t launch_fill_zero_u64(void* dst, int n, hipStream_t st);
// LDS bytes of the two block-forward kernels (for host-side validation).
size_t gemm_lds_bytes(int K, int mt = kMtBf16);
size_t prefill_lds_bytes(int hd);

// The current device's static scratch (kNoAllocScratchBytes, 256-byte aligned):
// its address is looked up once per device, on the first call with that device
// current.  Allocates nothing.
hipError_t noalloc_scratch(void** out);

// dst + b dst_stride <- src + b src_stride, row_bytes (a multiple of 16) each, b < B.
hipError_t launch_copy_rows(const void* src, size_t src_stride, void* dst, size_t dst_stride, size_t row_bytes, int B,
                            hipStream_t st);

// layout: the kvd_weight_layout of the weights (0 row-major, 1 packed, 2 packed
// with gamma folded in; 1 and 2 are bf16 only).
hipError_t launch_proj(const ProjArgs& a, int dtype_bf16, int hd, int layout, int n_units, hipStream_t st);
// Current-token projection (T == 1): the streaming kernel for bf16, proj_kernel for fp32.
hipError_t launch_project_current(const ProjArgs& a, int dtype_bf16, int hd, int layout, int n_units,
                                  hipStream_t st);
// engine: kFusedTile64 (fused_kernel), kFusedWide (the 128-token engine,
// fused_wide_kernel; bf16, head_dim 128 / 256, a.n_rec counted in 128-token
// tiles), kFusedSplit / kFusedSplit64 (fused_split_kernel; bf16, head_dim 128
// / 256, 128- or 64-token chunks, a tail of at most fold_rows rows, folded) or
// kFusedPair (fused_pair_kernel; bf16, head_dim 128, an even n_kv, two KV heads
// per 128-token tile, a.n_rec as on the wide engine).
enum { kFusedTile64 = 0, kFusedWide = 1, kFusedSplit = 2, kFusedSplit64 = 3, kFusedPair = 4 };
hipError_t launch_fused(const FusedArgs& a, int dtype_bf16, int hd, int layout, int engine, hipStream_t st);
// gamma: nullptr, or [d] bf16 folded into the packed values (bf16(w * gamma)).
hipError_t launch_pack(const void* w, const void* gamma, void* out, int rows, int d, hipStream_t st);
hipError_t launch_decode(const AttnArgs& a, int dtype_bf16, int hd, hipStream_t st);
hipError_t launch_combine(const float* ws_acc, const float* ws_ml, void* out, int n_q, int B, int S, int dtype_bf16,
                          int hd, hipStream_t st);

}  // namespace kvd
