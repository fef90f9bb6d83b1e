// Device building blocks of libkvd (gfx950 / CDNA4, wave64).
//
//  * stage_h:      one 8-element chunk of a residual row: gamma-scaled copy for
//                  the GEMM operand plus the row's sum of squares (RMSNorm,
//                  Sec. 3.1, Eqs. rmsnorm / rms_def).
//  * MfmaTile:     the bf16 recompute GEMM of one (token tile x 2*head_dim rows)
//                  block on v_mfma_f32_32x32x16_bf16: weights are the A operand
//                  (features = MFMA rows), the normalised residuals the B operand
//                  (tokens = MFMA columns), so each lane ends up holding whole RoPE
//                  pairs (2i, 2i+1) of one token.
//  * F32Tile:      the same contraction in fp32 on the vector ALUs.
//  * epilogues:    1/rms row scale, RoPE on key rows (Sec. 3.2, Eqs. rope_cos /
//                  rope_sin), one rounding to the storage type, into an LDS tile
//                  [tokens][K | V].
//  * attend_tile:  softmax partial state (max, sum, weighted V) of up to 64 keys
//                  of one KV head for its g query heads (Eqs. attn_weights /
//                  head_output, split over keys).
//
// Every path that produces K/V (prefill/recompute, current-token projection,
// fused kernel) runs the same tile code with the same K-loop order, the same
// sum-of-squares order and the same epilogue, which is what makes their K/V
// bit-identical (Prop. reconstruction: identical operation order).
#pragma once
#include <utility>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvd_layout.h"

namespace kvd {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int N> struct IC { static constexpr int value = N; };

// ------------------------------------------------------------------ scalars

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (round to nearest even) in one 32-bit word, a in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

__device__ __forceinline__ void load8(const uint16_t* p, float (&x)[8]) {
  uint4 v = *reinterpret_cast<const uint4*>(p);
  x[0] = bf_lo(v.x); x[1] = bf_hi(v.x); x[2] = bf_lo(v.y); x[3] = bf_hi(v.y);
  x[4] = bf_lo(v.z); x[5] = bf_hi(v.z); x[6] = bf_lo(v.w); x[7] = bf_hi(v.w);
}
__device__ __forceinline__ void load8(const float* p, float (&x)[8]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<uint16_t>(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ uint16_t from_f<uint16_t>(float v) {
  __bf16 x = (__bf16)v;
  return __builtin_bit_cast(uint16_t, x);
}
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }

// Wave-wide reductions on DPP lane moves (VALU only, no LDS round trips), in a
// fixed order: pairs and quads (quad_perm), 16-lane rows (row_ror 4, 8), then
// rows into lane 63 (row_bcast 15, 31); the result is broadcast from lane 63.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_mov(float old, float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old), __builtin_bit_cast(int, v),
                                                               CTRL, ROW_MASK, 0xf, false));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1, 0xf>(v, v));          // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_mov<0x4E, 0xf>(v, v));          // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_mov<0x124, 0xf>(v, v));         // row_ror 4
  v = fmaxf(v, dpp_mov<0x128, 0xf>(v, v));         // row_ror 8
  v = fmaxf(v, dpp_mov<0x142, 0xa>(-INFINITY, v)); // row_bcast 15
  v = fmaxf(v, dpp_mov<0x143, 0xc>(-INFINITY, v)); // row_bcast 31
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_mov<0xB1, 0xf>(v, v);
  v += dpp_mov<0x4E, 0xf>(v, v);
  v += dpp_mov<0x124, 0xf>(v, v);
  v += dpp_mov<0x128, 0xf>(v, v);
  v += dpp_mov<0x142, 0xa>(0.0f, v);
  v += dpp_mov<0x143, 0xc>(0.0f, v);
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// 1 / (log2(e)^-1 sqrt(head_dim)): scores are kept in the log2 domain.
template <int HD> struct ScoreScale;
template <> struct ScoreScale<64> { static constexpr float v = (float)(1.4426950408889634 / 8.0); };
template <> struct ScoreScale<128> { static constexpr float v = (float)(1.4426950408889634 / 11.313708498984761); };
template <> struct ScoreScale<256> { static constexpr float v = (float)(1.4426950408889634 / 16.0); };

// RoPE rotation of one pair by +p*omega_i, omega_i = 2*pi*rev (rev in
// revolutions per position).  The angle is reduced in fp64 so that large
// positions keep full fp32 accuracy; the hardware sine/cosine take revolutions.
__device__ __forceinline__ void rope_rotate(float& x0, float& x1, int p, double rev) {
  double a = (double)p * rev;
  a -= rint(a);
  const float t = (float)a;
  const float sn = __builtin_amdgcn_sinf(t);
  const float cs = __builtin_amdgcn_cosf(t);
  const float y0 = fmaf(x0, cs, -(x1 * sn));
  const float y1 = fmaf(x0, sn, x1 * cs);
  x0 = y0;
  x1 = y1;
}

// ------------------------------------------------------------------ residual staging

// One 8-element chunk of a residual row: accumulate sum(h^2) in element order and
// return bf16(h * gamma).
__device__ __forceinline__ uint4 stage_chunk_bf16(uint4 hv, uint4 gv, float& ss) {
  const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
  const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float h0 = bf_lo(hw[i]), h1 = bf_hi(hw[i]);
    ss = fmaf(h0, h0, ss);
    ss = fmaf(h1, h1, ss);
    o[i] = pack_bf16x2(h0 * bf_lo(gw[i]), h1 * bf_hi(gw[i]));
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

// The two halves of stage_chunk_bf16, with the same arithmetic: the sum of squares
// of one chunk in element order, and bf16(h * gamma) of one chunk.
__device__ __forceinline__ void sumsq_chunk_bf16(uint4 hv, float& ss) {
  const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float h0 = bf_lo(hw[i]), h1 = bf_hi(hw[i]);
    ss = fmaf(h0, h0, ss);
    ss = fmaf(h1, h1, ss);
  }
}
__device__ __forceinline__ uint4 scale_chunk_bf16(uint4 hv, uint4 gv) {
  const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
  const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = pack_bf16x2(bf_lo(hw[i]) * bf_lo(gw[i]), bf_hi(hw[i]) * bf_hi(gw[i]));
  return make_uint4(o[0], o[1], o[2], o[3]);
}

// Folded weights (W diag(gamma), kvd_pack_weights_gamma): the residual chunk is
// staged unchanged and its sum of squares takes one dot2 per word (both
// products exact in fp32, added to the running sum).  Every producer of folded
// K/V runs this chain per (token, 8-element column chunk) in K order, so they
// stay bit-identical to each other.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void sumsq_chunk_dot2(uint4 hv, float& ss) {
  ss = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, hv.x), __builtin_bit_cast(bf16x2_t, hv.x), ss, false);
  ss = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, hv.y), __builtin_bit_cast(bf16x2_t, hv.y), ss, false);
  ss = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, hv.z), __builtin_bit_cast(bf16x2_t, hv.z), ss, false);
  ss = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, hv.w), __builtin_bit_cast(bf16x2_t, hv.w), ss, false);
}
// The staged B-operand chunk and the sum of squares, for weights with gamma
// applied by the kernel (FOLD = false: bf16(gamma * h)) or folded into them.
template <bool FOLD>
__device__ __forceinline__ uint4 stage_chunk(uint4 hv, uint4 gv, float& ss) {
  if constexpr (FOLD) {
    sumsq_chunk_dot2(hv, ss);
    return hv;
  } else {
    return stage_chunk_bf16(hv, gv, ss);
  }
}
template <bool FOLD>
__device__ __forceinline__ void sumsq_chunk(uint4 hv, float& ss) {
  if constexpr (FOLD) sumsq_chunk_dot2(hv, ss);
  else sumsq_chunk_bf16(hv, ss);
}

// Per-token 1/rms from the per-thread partial sums: thread (row, sub) holds the
// sum over its chunk column sub = tid & 7; the 8 partials of a row sit in 8
// consecutive lanes and are added by a fixed xor tree.  Rows of thread tid are
// (tid >> 3) + (NT / 8) * r.
template <int NT, int CPT>
__device__ __forceinline__ void finish_rms(const float (&ss)[CPT], const bool (&valid)[CPT], int d, float eps,
                                           float* rinv) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int r = 0; r < CPT; ++r) {
    float v = ss[r];
    v += __shfl_xor(v, 1, 64);
    v += __shfl_xor(v, 2, 64);
    v += __shfl_xor(v, 4, 64);
    if ((tid & 7) == 0) rinv[(tid >> 3) + (NT / 8) * r] = valid[r] ? 1.0f / sqrtf(v / (float)d + eps) : 0.0f;
  }
}

// One half (head_dim rows) of a projection tile: the weight block it reads and
// whether its rows get RoPE.  Column offset in the LDS K/V tile: half * head_dim.
struct Half {
  const void* w;  // first row of a [head_dim][d] block, or nullptr (rows absent -> zeros)
  int rope;
};

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// s_waitcnt immediate that waits until at most n (< 64) vector memory operations
// of the wave are outstanding (expcnt and lgkmcnt left unconstrained).
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0f70; }

// Slot (16 bytes) of B-fragment lane lam (0..63; column lam % 32, k-half lam / 32)
// of substep u inside its 1 KiB staged fragment.  Staging thread (token row,
// column chunk sub) writes fragment sub / 2, lane row % 32 + 32 (sub % 2): the
// 8 lanes of one token would all land on the same LDS banks in lane order,
// eight-way conflicts on every staging write.  The XOR below spreads them (and
// any 8 or 16 consecutive lanes of a write or of a fragment read) over distinct
// banks; only addresses change, never an operand.
__device__ __forceinline__ int bslot(int lam, int u) { return lam ^ (u << 1) ^ ((lam >> 5) * 9); }

// Element offset of the MFMA A operand chunk (K-step s, 16-wide substep u) from a
// lane's base pointer.  Row-major: base = row (row0 + lane % 32), column 8 (lane / 32);
// packed (kvd_pack_weights): base = block row row0 + lane * 8, one 512-element
// block per 16 columns.
template <bool PACKED>
__device__ __forceinline__ size_t w_off(int s, int u) {
  return PACKED ? ((size_t)s * (kKT / 16) + u) * 512 : (size_t)s * kKT + 16 * u;
}

// ------------------------------------------------------------------ bf16 MFMA tile

// 8 waves (512 threads) compute a [2*HD features] x [MT tokens] tile.  Waves are
// arranged WF (features) x WT (tokens); each owns NB_F 32-row blocks and NB_T
// 32-token blocks.  head_dim 256: every wave owns 32 K rows and the same 32 V
// rows (RoPE work balanced); head_dim 128 / 64: waves own one 32-row block of
// either half.  Weights stream from global memory straight into MFMA A-operand
// registers (each weight byte is used by exactly one wave), kDepth K-steps
// ahead; gamma-scaled residuals are staged through LDS (shared by all waves),
// double buffered.
template <int HD, int MT, bool PACKED, bool FOLD = false>
struct MfmaTile {
  static constexpr int NT = kNtTile;
  static constexpr int NW = NT / 64;
  static constexpr int WF = HD == 64 ? 4 : 8;
  static constexpr int WT = NW / WF;
  static constexpr int NB_F = (2 * HD / WF) / 32;
  static constexpr int TOK_W = MT / WT;
  static constexpr int NB_T = TOK_W / 32;
  static constexpr int CPT = MT * 8 / NT;  // staged 8-element chunks per thread per K-step
  static constexpr int HLD = h_ld<uint16_t>();
  static constexpr int KLD = kv_ld<uint16_t>(HD);
  static_assert(NB_F >= 1 && NB_T >= 1 && CPT >= 1, "tile shape");

  static __device__ __forceinline__ void block_rows(int fw, int bf, int& half, int& row0) {
    if (NB_F == 2) {
      half = bf;
      row0 = 32 * fw;
    } else {
      half = fw / (WF / 2);
      row0 = 32 * (fw % (WF / 2));
    }
  }

  // Computes the tile into `kv` (LDS, [MT][KLD] bf16).  hrow[r]: residual row of
  // staged token (tid>>3)+64r, offset by 8*(tid&7) (any readable row if !valid[r]).
  // gam: gamma in LDS ([d] bf16), gam_g: the same in global memory.  setup():
  // the caller's LDS writes of gam, pos and rev (and anything else it needs),
  // run after the K-loop's first loads are issued so that the latency of the
  // caller's own loads overlaps theirs; no barrier may precede it.
  template <class Setup>
  static __device__ __forceinline__ void run(const uint16_t* const (&hrow)[CPT], const bool (&valid)[CPT], const uint16_t* gam,
                             const uint16_t* gam_g, int d, float eps, const Half (&halves)[2], uint16_t* hst,
                             float* rinv, const int* pos, const double* rev, uint16_t* kv, const Setup& setup) {
    const int rope0 = halves[0].rope, rope1 = halves[1].rope;
    run_with(hrow, valid, gam, gam_g, d, eps, halves, hst, rinv, setup,
             [&](const f32x16_t (&acc)[NB_F][NB_T], const bool (&wok)[NB_F]) {
               store_kv(acc, wok, rope0, rope1, rinv, pos, rev, kv);
             });
  }

  // Epilogue of run(): row scale, RoPE on rotated halves, one RNE rounding, LDS tile.
  static __device__ __forceinline__ void store_kv(const f32x16_t (&acc)[NB_F][NB_T], const bool (&wok)[NB_F],
                                                  int rope0, int rope1, const float* rinv, const int* pos,
                                                  const double* rev, uint16_t* kv) {
    const int lane = threadIdx.x & 63, wave = wave_id();
    const int fw = wave % WF, tw = wave / WF;
#pragma unroll
    for (int bt = 0; bt < NB_T; ++bt) {
      const int tok = tw * TOK_W + 32 * bt + (lane & 31);
      const float ri = rinv[tok];
      const int p = pos[tok];
#pragma unroll
      for (int bf = 0; bf < NB_F; ++bf) {
        int half, row0;
        block_rows(fw, bf, half, row0);
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = wok[bf] ? acc[bf][bt][r] * ri : 0.0f;
        if (half ? rope1 : rope0) {
#pragma unroll
          for (int r = 0; r < 16; r += 2) {
            const int f = row0 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            rope_rotate(v[r], v[r + 1], p, rev[f >> 1]);
          }
        }
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int col = half * HD + row0 + 8 * g4 + 4 * (lane >> 5);
          uint2 o;
          o.x = pack_bf16x2(v[4 * g4 + 0], v[4 * g4 + 1]);
          o.y = pack_bf16x2(v[4 * g4 + 2], v[4 * g4 + 3]);
          *reinterpret_cast<uint2*>(kv + (size_t)tok * KLD + col) = o;
        }
      }
    }
  }

  // The K-loop and the tokens' 1/rms (in rinv), then epi(acc, wok) with the
  // fp32 accumulators: acc[bf][bt][r] is feature row0(bf) + 8 (r / 4) +
  // 4 (lane / 32) + r % 4 of half(bf) (block_rows) for token tw TOK_W + 32 bt +
  // lane % 32, wok[bf] whether that half's weights are present.
  template <class Setup, class Epi>
  static __device__ __forceinline__ void run_with(const uint16_t* const (&hrow)[CPT], const bool (&valid)[CPT],
                                                  const uint16_t* gam, const uint16_t* gam_g, int d, float eps,
                                                  const Half (&halves)[2], uint16_t* hst, float* rinv,
                                                  const Setup& setup, const Epi& epi) {
    const int tid = threadIdx.x, lane = tid & 63, sub = tid & 7;
    const int wave = wave_id();
    const int fw = wave % WF, tw = wave / WF;
    const int nsteps = d / kKT;

    // the halves' weight pointers as values (a runtime choice between two array
    // elements would keep the array in scratch memory)
    const void* const hw0 = halves[0].w;
    const void* const hw1 = halves[1].w;
    const uint16_t* wrow[NB_F];
    bool wok[NB_F];
#pragma unroll
    for (int bf = 0; bf < NB_F; ++bf) {
      int half, row0;
      block_rows(fw, bf, half, row0);
      const uint16_t* w = static_cast<const uint16_t*>(half ? hw1 : hw0);
      wok[bf] = w != nullptr;  // uniform per wave
      const uint16_t* wb = wok[bf] ? w : static_cast<const uint16_t*>(hw0);
      wrow[bf] = PACKED ? wb + (size_t)row0 * d + 8 * lane
                        : wb + (size_t)(row0 + (lane & 31)) * d + 8 * (lane >> 5);
    }

    f32x16_t acc[NB_F][NB_T];
#pragma unroll
    for (int bf = 0; bf < NB_F; ++bf)
#pragma unroll
      for (int bt = 0; bt < NB_T; ++bt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[bf][bt][i] = 0.0f;

    // K-loop.  Weights: a ring of D = 4 K-steps in A-operand registers, each
    // 16-wide substep refilled right after its MFMAs.  Residuals: loaded D - 1
    // steps ahead into registers, staged (gamma * h -> bf16, sum of squares) one
    // step ahead into an LDS ring of D slots laid out in MFMA B-fragment order
    // (fragment f = 4 * token block + substep, 64 lanes x 8 elements), so every
    // wave reads its B operands as contiguous 1 KB blocks.  One barrier per step,
    // in its middle: before it the step's first two substeps; after it the next
    // step's fragments are valid, so the next step's first fragments are read
    // during the last two substeps.  Per accumulator the MFMA chain is in K order.
    static_assert(CPT == 1 && MT == 64, "one staged chunk per thread, two 32-token blocks");
    constexpr int D = 4;
    constexpr int SLOT = 8 * 512;  // elements per LDS slot
    bf16x8_t A[D][NB_F][4];
    uint4 H[D];
    float ss[CPT] = {0.0f};
    const int row = tid >> 3;
    const int lofs = ((row >> 5) * 4 + (sub >> 1)) * 512 + 8 * bslot((row & 31) + 32 * (sub & 1), sub >> 1);
    const int bt0 = NB_T == 2 ? 0 : tw;  // first absolute token block of this wave

    auto load_wu = [&](int slot, int s, int u) {
#pragma unroll
      for (int bf = 0; bf < NB_F; ++bf)
        A[slot][bf][u] = *reinterpret_cast<const bf16x8_t*>(wrow[bf] + w_off<PACKED>(s, u));
    };
    auto load_h = [&](int slot, int s) { H[slot] = *reinterpret_cast<const uint4*>(hrow[0] + (size_t)s * kKT); };
    // Tokens past the end of a ragged tile stage a readable row's values: their
    // MFMA columns are independent of the others and their 1/rms is zero.
    auto put_hv = [&](int slot, const uint4& gv) {
      *reinterpret_cast<uint4*>(hst + (size_t)slot * SLOT + lofs) = stage_chunk<FOLD>(H[slot], gv, ss[0]);
    };
    auto put_h = [&](int slot, int s) {
      put_hv(slot, FOLD ? uint4{} : *reinterpret_cast<const uint4*>(gam + (size_t)s * kKT + 8 * sub));
    };
    auto rd = [&](bf16x8_t (&bv)[NB_T], int slot, int u) {
#pragma unroll
      for (int bt = 0; bt < NB_T; ++bt)
        bv[bt] = *reinterpret_cast<const bf16x8_t*>(hst + (size_t)slot * SLOT + ((bt0 + bt) * 4 + u) * 512 +
                                                    8 * bslot(lane, u));
    };
    auto mma = [&](int slot, int u, const bf16x8_t (&bv)[NB_T]) {
#pragma unroll
      for (int bf = 0; bf < NB_F; ++bf)
#pragma unroll
        for (int bt = 0; bt < NB_T; ++bt)
          acc[bf][bt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[slot][bf][u], bv[bt], acc[bf][bt], 0, 0, 0);
    };
    // interleave of one substep: its B reads, then MFMAs and weight refills alternating
    auto sched_substep = [&]() {
      __builtin_amdgcn_sched_group_barrier(0x100, NB_T, 0);  // DS read
#pragma unroll
      for (int i = 0; i < NB_F; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, NB_T, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);     // VMEM read
      }
    };
    bf16x8_t b0[NB_T];
    // iteration s (slot L = s % D): GUARD = false for the steady state (every
    // step index below is in range), true for the last iterations.
    auto iter = [&](auto lc, int s, auto guard_c) {
      constexpr int L = decltype(lc)::value;
      constexpr bool GUARD = decltype(guard_c)::value;
      const int sw = GUARD ? min(s + D, nsteps - 1) : s + D;
      __builtin_amdgcn_sched_barrier(0);
      if (!GUARD || s + 1 < nsteps) put_h((L + 1) % D, s + 1);
      bf16x8_t b1[NB_T], b2[NB_T], b3[NB_T];
      rd(b1, L, 1);
      mma(L, 0, b0);
      load_wu(L, sw, 0);
      mma(L, 1, b1);
      load_wu(L, sw, 1);
      if (!GUARD) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // gamma
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // staged chunk
        __builtin_amdgcn_sched_group_barrier(0x100, NB_T, 0);
#pragma unroll
        for (int i = 0; i < NB_F; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, NB_T, 0);
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        }
#pragma unroll
        for (int i = 0; i < NB_F; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, NB_T, 0);
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's staged chunk is in LDS
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      rd(b2, L, 2);
      rd(b3, L, 3);
      load_h(L, GUARD ? min(s + D, nsteps - 1) : s + D);
      mma(L, 2, b2);
      load_wu(L, sw, 2);
      rd(b0, (L + 1) % D, 0);
      mma(L, 3, b3);
      load_wu(L, sw, 3);
      if (!GUARD) {
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * NB_T, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // residual load
        sched_substep();
        sched_substep();
      }
    };

    // prologue: residual steps 0..D-1 and weight steps 0..D-1 in flight, the
    // caller's setup written, step 0 staged (its gamma chunk read from global
    // memory: the LDS copy is complete only after the barrier)
#pragma unroll
    for (int i = 0; i < D; ++i) load_h(i, min(i, nsteps - 1));
    const uint4 g0 = FOLD ? uint4{} : *reinterpret_cast<const uint4*>(gam_g + 8 * sub);
    __builtin_amdgcn_sched_barrier(0);  // keep it ahead of the weight loads (in-order waits)
#pragma unroll
    for (int i = 0; i < D; ++i)
#pragma unroll
      for (int u = 0; u < 4; ++u) load_wu(i, min(i, nsteps - 1), u);
    setup();
    put_hv(0, g0);
    load_h(0, min(D, nsteps - 1));
    __syncthreads();
    rd(b0, 0, 0);
    int s0 = 0;
    // steady state: iterations s0..s0+3 all have s + D < nsteps
    for (; s0 + 2 * D <= nsteps; s0 += D) {
      iter(IC<0>{}, s0, IC<0>{});
      iter(IC<1>{}, s0 + 1, IC<0>{});
      iter(IC<2>{}, s0 + 2, IC<0>{});
      iter(IC<3>{}, s0 + 3, IC<0>{});
    }
    for (; s0 < nsteps; s0 += D) {
      iter(IC<0>{}, s0, IC<1>{});
      if (s0 + 1 < nsteps) iter(IC<1>{}, s0 + 1, IC<1>{});
      if (s0 + 2 < nsteps) iter(IC<2>{}, s0 + 2, IC<1>{});
      if (s0 + 3 < nsteps) iter(IC<3>{}, s0 + 3, IC<1>{});
    }
    __syncthreads();

    finish_rms<NT, CPT>(ss, valid, d, eps, rinv);
    __syncthreads();

    epi(acc, wok);
  }
};

// ------------------------------------------------------------------ bf16 MFMA tile, 128 tokens

// 8 waves (512 threads, two per SIMD) compute a [2*HD features] x [MT tokens]
// tile (MT = 128, or 64 for grids too small for 128-token tiles), head_dim 128
// or 256.  Wave w owns 32 feature rows for all MT tokens per 32-row block it
// holds: at head_dim 256 K rows and the same V rows
// [32 w, 32 w + 32) (two blocks, RoPE work balanced), at head_dim 128 one block
// of K (waves 0-3) or V (waves 4-7).  Each weight (A) fragment feeds one MFMA
// per 32-token block.  With MT = 128 a CU reads the tile's weights once per 128
// tokens instead of once per 64 (half the weight bytes per flop of MfmaTile),
// and the two waves of a SIMD cover each other's staging arithmetic, fragment
// reads and barrier waits.  The per-element arithmetic is MfmaTile's: the same
// MFMA chain over d in K order, the same staging, 1/rms and epilogue, so the
// K/V it produces are bit-identical.
//
// Split layout (NTX = kNtSplit: 4 waves, one per SIMD): the tile is one half
// only, the HD rows of halves[0] (a KV head's K rows or its V rows) for MT
// tokens; wave w owns rows [32 NB_F w, 32 NB_F (w + 1)).  Per wave the work is
// the 8-wave layout's (NB_F row blocks for all MT tokens), so a CU streams the
// half's weights once per MT tokens: at MT = 128 half the weight bytes per flop
// of a 64-token tile of both halves, over the same number of workgroups.  The
// K/V tile then holds the half's HD columns only (row stride KLDX).
//
// K-loop: weights are loaded DW = 2 K-steps ahead into A-operand registers,
// each substep's fragments refilled right after its MFMAs; residuals one step
// ahead into registers, staged (gamma * h -> bf16, sum of squares) two steps
// ahead into an LDS ring of kDepth slots in B-fragment order.  One barrier
// per step, after the second substep.  Loads go through
// buffer resources (wave-uniform base and extent in SGPRs, a 32-bit offset per
// lane), which keeps the addresses out of the vector registers.
// RLEAD (tiles of both halves): residual rows two K-steps ahead and weights one
// (instead of one and two), for the same register count; taken by the callers
// whose tiles it measured faster (the block GEMMs, the KV-head pairs, the
// 64-token fused tiles, the wide prefill), not by the wide fused engine.
template <int HD, int MT, bool PACKED, bool FOLD = false, int NTX = kNtWide, int KLDX = kv_ld<uint16_t>(HD),
          bool SPLITX = false, bool RLEAD = false>
struct WideTile {
  static constexpr int NT = NTX;
  static constexpr int NW = NT / 64;
  static constexpr bool SPLIT = SPLITX;   // one half per tile
  static constexpr int NB_F = SPLIT ? HD / (32 * NW) : HD / 128;   // 32-row blocks per wave
  static constexpr int NB_T = MT / 32;    // 32-token blocks (all of them)
  static constexpr int CPT = MT * 8 / NT;  // staged 8-element chunks per thread per K-step
  static constexpr int TPR = NT / 8;       // tokens staged per chunk index (one per 8 threads)
  static constexpr int KLD = KLDX;
  // weight K-steps in flight: a split wave of one 32-row block holds 4 (its
  // A fragments are half the 8-wave layout's per step)
  static constexpr int DW = SPLIT && NB_F == 1 ? 4 : (RLEAD ? 1 : 2);
  // residual K-steps in registers: a split wave of one 32-row block has so
  // little work per K-step that one step of lead does not cover the load
  // latency, so it keeps two steps in flight, and four on 64-token tiles
  // (half the work per step again; its registers allow it without spills)
  static constexpr int DH = SPLIT && NB_F == 1 ? (MT == 64 ? 4 : 2) : (RLEAD ? 2 : 1);
  static_assert(!RLEAD || !SPLIT, "RLEAD: tiles of both halves");
  static constexpr int DL = kDepth;
  static constexpr int SLOT = NB_T * 4 * 512;  // elements per LDS slot (one K-step)
  static constexpr int NU = 4 * NB_T;          // units (substep, token block) per K-step
  // VALU instructions the schedule interleaves after each MFMA of the first
  // half-step (the staging arithmetic of CPT chunks per thread)
  static constexpr int VPM = SPLIT ? 5 * CPT / NB_F : 5;
  static_assert(HD == 128 || HD == 256, "wide tile: head_dim 128 or 256");
  static_assert((MT == 64 || MT == 128) && DL == 4 && CPT * NT == MT * 8 && (NT == 512 || NT == 256) &&
                    TPR % 32 == 0 && CPT >= 1 && NB_F >= 1 && (!SPLIT || NB_F * 32 * NW == HD),
                "ring and staging shape");

  static __device__ __forceinline__ void block_rows(int w, int bf, int& half, int& row0) {
    if (SPLIT) {
      half = 0;
      row0 = 32 * (NB_F * w + bf);
    } else if (NB_F == 2) {
      half = bf;
      row0 = 32 * w;
    } else {
      half = w / 4;
      row0 = 32 * (w % 4);
    }
  }

  // As MfmaTile::run, for the n <= MT residual rows that start at h_tile
  // ([n][d], row stride d); the K/V tile goes to `kv`.
  template <class Setup>
  static __device__ __forceinline__ void run(const uint16_t* h_tile, int n, const uint16_t* gam, const uint16_t* gam_g,
                                             int d, float eps, const Half (&halves)[2], uint16_t* hst, float* rinv,
                                             const int* pos, const double* rev, uint16_t* kv, const Setup& setup) {
    const int rope0 = halves[0].rope, rope1 = halves[1].rope;
    run_with(h_tile, n, gam, gam_g, d, eps, halves, hst, rinv, setup,
             [&](const f32x16_t (&acc)[NB_F][NB_T], const bool (&wok)[NB_F]) {
               store_kv(acc, wok, rope0, rope1, rinv, pos, rev, kv);
             });
  }

  // MfmaTile::store_kv for this wave layout.
  static __device__ __forceinline__ void store_kv(const f32x16_t (&acc)[NB_F][NB_T], const bool (&wok)[NB_F],
                                                  int rope0, int rope1, const float* rinv, const int* pos,
                                                  const double* rev, uint16_t* kv) {
    const int lane = threadIdx.x & 63, w = wave_id();
#pragma unroll
    for (int bt = 0; bt < NB_T; ++bt) {
      const int tok = 32 * bt + (lane & 31);
      const float ri = rinv[tok];
      const int p = pos[tok];
#pragma unroll
      for (int bf = 0; bf < NB_F; ++bf) {
        int half, row0;
        block_rows(w, bf, half, row0);
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = wok[bf] ? acc[bf][bt][r] * ri : 0.0f;
        if (half ? rope1 : rope0) {
#pragma unroll
          for (int r = 0; r < 16; r += 2) {
            const int f = row0 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            rope_rotate(v[r], v[r + 1], p, rev[f >> 1]);
          }
        }
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int col = half * HD + row0 + 8 * g4 + 4 * (lane >> 5);
          uint2 o;
          o.x = pack_bf16x2(v[4 * g4 + 0], v[4 * g4 + 1]);
          o.y = pack_bf16x2(v[4 * g4 + 2], v[4 * g4 + 3]);
          *reinterpret_cast<uint2*>(kv + (size_t)tok * KLD + col) = o;
        }
      }
    }
  }

  // The K-loop and 1/rms (in rinv), then epi(acc, wok): acc[bf][bt][r] is
  // feature row0(bf) + 8 (r / 4) + 4 (lane / 32) + r % 4 of half(bf) for token
  // 32 bt + lane % 32.
  template <class Setup, class Epi>
  static __device__ __forceinline__ void run_with(const uint16_t* h_tile, int n, const uint16_t* gam,
                                                  const uint16_t* gam_g, int d, float eps, const Half (&halves)[2],
                                                  uint16_t* hst, float* rinv, const Setup& setup, const Epi& epi) {
    const int tid = threadIdx.x, lane = tid & 63, sub = tid & 7;
    const int w = wave_id();
    const int nsteps = d / kKT;

    // weights: this wave's 32 rows of each block; a half without weights reads
    // the other half's rows (in bounds) and its results are zeros
    const void* const hw0 = halves[0].w;
    const void* const hw1 = halves[1].w;
    const void* const wk = hw0 != nullptr ? hw0 : hw1;
    const void* const wv = hw1 != nullptr ? hw1 : wk;
    bool wok[NB_F];
    __amdgpu_buffer_rsrc_t wres[NB_F];
#pragma unroll
    for (int bf = 0; bf < NB_F; ++bf) {
      int half, row0;
      block_rows(w, bf, half, row0);
      wok[bf] = (half ? hw1 : hw0) != nullptr;  // uniform per wave
      const uint16_t* wp = static_cast<const uint16_t*>(half ? wv : wk) + (size_t)row0 * d;
      wres[bf] = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(wp), (short)0, (int)(32u * (uint32_t)d * 2u),
                                                   0x00020000);
    }
    // byte offset of this lane's A-operand chunk at K-step 0, substep 0
    const uint32_t wlane = PACKED ? 16u * lane : 2u * ((uint32_t)(lane & 31) * d + 8u * (lane >> 5));
    // residuals: rows (tid >> 3) + 64 r; rows past n read row 0 (their MFMA
    // columns are independent of the others and their 1/rms is zero)
    bool valid[CPT];
    uint32_t hoff[CPT];
    const __amdgpu_buffer_rsrc_t hres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(h_tile), (short)0, (int)((uint32_t)n * (uint32_t)d * 2u), 0x00020000);
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
      const int t = (tid >> 3) + TPR * r;
      valid[r] = t < n;
      hoff[r] = 2u * ((uint32_t)(valid[r] ? t : 0) * (uint32_t)d + 8u * sub);
    }

    f32x16_t acc[NB_F][NB_T];
#pragma unroll
    for (int bf = 0; bf < NB_F; ++bf)
#pragma unroll
      for (int bt = 0; bt < NB_T; ++bt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[bf][bt][i] = 0.0f;
    // The accumulators live in AGPRs (the MFMAs' AGPR form): an empty asm
    // statement that names them with the AGPR constraint tells the compiler
    // this wave uses AGPRs, which leaves the 128 VGPRs to the operand rings.
#pragma unroll
    for (int bf = 0; bf < NB_F; ++bf)
#pragma unroll
      for (int bt = 0; bt < NB_T; ++bt) asm volatile("" : "+a"(acc[bf][bt]));

    bf16x8_t A[DW][NB_F][4];
    uint4 H[DH][CPT];
    float ss[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) ss[r] = 0.0f;
    // chunk r of this thread: token (tid >> 3) + TPR r = token block
    // (tid >> 8) + (TPR / 32) r, column (tid >> 3) % 32; elements 8 sub .. 8 sub + 7 of
    // the K-step = substep sub / 2, lane half sub % 2 of the B fragment
    const int lofs = ((tid >> 8) * 4 + (sub >> 1)) * 512 + 8 * bslot(((tid >> 3) & 31) + 32 * (sub & 1), sub >> 1);

    auto load_wu = [&](int slot, int s, int u) {
#pragma unroll
      for (int bf = 0; bf < NB_F; ++bf) {
        const u32x4_t v =
            __builtin_amdgcn_raw_buffer_load_b128(wres[bf], (int)wlane, (int)(2u * (uint32_t)w_off<PACKED>(s, u)), 0);
        A[slot][bf][u] = __builtin_bit_cast(bf16x8_t, v);
      }
    };
    auto load_h = [&](int hslot, int s) {
#pragma unroll
      for (int r = 0; r < CPT; ++r) {
        const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(hres, (int)hoff[r], 2 * s * kKT, 0);
        H[hslot][r] = make_uint4(v.x, v.y, v.z, v.w);
      }
    };
    auto put_hv = [&](int lslot, int hslot, const uint4& gv) {
#pragma unroll
      for (int r = 0; r < CPT; ++r)
        *reinterpret_cast<uint4*>(hst + (size_t)lslot * SLOT + r * (TPR / 32) * 4 * 512 + lofs) =
            stage_chunk<FOLD>(H[hslot][r], gv, ss[r]);
    };
    // B fragment of K-step slot lslot, substep u, token block bt
    auto rd1 = [&](int lslot, int u, int bt) {
      return *reinterpret_cast<const bf16x8_t*>(hst + (size_t)lslot * SLOT + (bt * 4 + u) * 512 + 8 * bslot(lane, u));
    };

    // A step is NU units k = NB_T u + bt (substep u, token block bt), each one B
    // fragment and the NB_F MFMAs that use it.  B fragments stream through a
    // ring of RA + 1 registers, read RA units ahead: the reads of the next
    // step's first units come after the barrier (after unit NU / 2 - 1) that
    // makes its staging visible.
    constexpr int RA = 3;
    constexpr int NBQ = RA + 1;
    static_assert(NU % NBQ == 0 && RA < NU / 2, "unit k of every step uses ring entry k % NBQ");
    bf16x8_t bq[NBQ];
    // iteration s, L = s % 4: weight slot s % 2 (refilled with step s + 2), the
    // residual registers (staged as step s + 1, then refilled with step s + 2),
    // LDS slot L (read) and (L + 1) % 4 (written).  GUARD: the last iterations,
    // whose step indexes are clamped into range.  Units keep their order (a
    // scheduling fence after each lets only VALU, SALU, DS writes and
    // transcendentals cross), so every ring register is reloaded only after its
    // last use, and the staging arithmetic spreads over the first half.
    auto iter = [&](auto lc, int s, auto guard_c) {
      constexpr int L = decltype(lc)::value;
      constexpr int LW = L % DW;
      constexpr int LN = (L + 1) & 3;
      constexpr bool GUARD = decltype(guard_c)::value;
      const int sw = GUARD ? min(s + DW, nsteps - 1) : s + DW;
      const int sh = GUARD ? min(s + 1 + DH, nsteps - 1) : s + 1 + DH;
      auto unit = [&](auto kc) {
        constexpr int k = decltype(kc)::value;
        constexpr int u = k / NB_T, bt = k % NB_T, kk = k + RA;
        if constexpr (kk < NU) bq[kk % NBQ] = rd1(L, kk / NB_T, kk % NB_T);
        else bq[kk % NBQ] = rd1(LN, (kk - NU) / NB_T, (kk - NU) % NB_T);
#pragma unroll
        for (int bf = 0; bf < NB_F; ++bf)
          acc[bf][bt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[LW][bf][u], bq[k % NBQ], acc[bf][bt], 0, 0, 0);
        if constexpr (bt == NB_T - 1) load_wu(LW, sw, u);
        if constexpr (k == NB_T - 1) load_h((L + 1) % DH, sh);
        if (!GUARD) {
          __builtin_amdgcn_sched_group_barrier(0x100, k == 0 ? 2 : 1, 0);  // DS read: B fragment (gamma)
#pragma unroll
          for (int bf = 0; bf < NB_F; ++bf) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);            // MFMA
            if constexpr (k < NU / 2 - 1) __builtin_amdgcn_sched_group_barrier(0x002, VPM, 0);  // VALU: staging
          }
          if constexpr (k == NU / 2 - 2) __builtin_amdgcn_sched_group_barrier(0x200, CPT, 0);  // DS write: staged chunks
        }
        __builtin_amdgcn_sched_barrier(0x0606);
      };
      __builtin_amdgcn_sched_barrier(0);
      if (!GUARD || s + 1 < nsteps)
        put_hv(LN, (L + 1) % DH, FOLD ? uint4{} : *reinterpret_cast<const uint4*>(gam + (size_t)(s + 1) * kKT + 8 * sub));
      [&]<int... K>(std::integer_sequence<int, K...>) { (unit(IC<K>{}), ...); }(std::make_integer_sequence<int, NU / 2>{});
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's staged chunks are in LDS
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      [&]<int... K>(std::integer_sequence<int, K...>) {
        (unit(IC<K + NU / 2>{}), ...);
      }(std::make_integer_sequence<int, NU / 2>{});
    };

    // prologue: residual step 0 and weight steps 0, 1 in flight, the caller's
    // setup written, step 0 staged (its gamma chunk read from global memory:
    // the LDS copy is complete only after the barrier), step 1's residuals
    // requested
    load_h(0, 0);
    const uint4 g0 = FOLD ? uint4{} : *reinterpret_cast<const uint4*>(gam_g + 8 * sub);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < DW; ++i)
#pragma unroll
      for (int u = 0; u < 4; ++u) load_wu(i, min(i, nsteps - 1), u);
    setup();
    put_hv(0, 0, g0);
    // steps 1 .. DH into slots 1 % DH .. DH % DH
#pragma unroll
    for (int i = 1; i <= DH; ++i) load_h(i % DH, min(i, nsteps - 1));
    __syncthreads();
#pragma unroll
    for (int k = 0; k < RA; ++k) bq[k] = rd1(0, k / NB_T, k % NB_T);
    int s0 = 0;
    // steady state: every step index of iterations s0 .. s0 + 3 is below nsteps
    for (; s0 + 8 <= nsteps; s0 += 4) {
      iter(IC<0>{}, s0, IC<0>{});
      iter(IC<1>{}, s0 + 1, IC<0>{});
      iter(IC<2>{}, s0 + 2, IC<0>{});
      iter(IC<3>{}, s0 + 3, IC<0>{});
    }
    for (; s0 < nsteps; s0 += 4) {
      iter(IC<0>{}, s0, IC<1>{});
      if (s0 + 1 < nsteps) iter(IC<1>{}, s0 + 1, IC<1>{});
      if (s0 + 2 < nsteps) iter(IC<2>{}, s0 + 2, IC<1>{});
      if (s0 + 3 < nsteps) iter(IC<3>{}, s0 + 3, IC<1>{});
    }
    __syncthreads();

    finish_rms<NT, CPT>(ss, valid, d, eps, rinv);
    __syncthreads();

    epi(acc, wok);
  }
};

// ------------------------------------------------------------------ fp32 VALU tile

// The same contraction in fp32 on the vector ALUs: thread (pair p, token group)
// accumulates rows 2p, 2p+1 of the 2*HD rows for TPT tokens, in d order.
template <int HD, int MT>
struct F32Tile {
  static constexpr int NT = kNtTile;
  static constexpr int TG = NT / HD;         // token groups
  static constexpr int TPT = MT / TG;        // tokens per thread
  static constexpr int CPT = MT * 8 / NT;
  static constexpr int HLD = h_ld<float>();
  static constexpr int KLD = kv_ld<float>(HD);

  // setup(): the caller's LDS writes of pos and rev (read after the K-loop's
  // barriers), run first.
  template <class Setup>
  static __device__ __forceinline__ void run(const float* const (&hrow)[CPT], const bool (&valid)[CPT], const float* gamma, int d,
                             float eps, const Half (&halves)[2], float* hst, float* rinv, const int* pos,
                             const double* rev, float* kv, const Setup& setup) {
    setup();
    const int tid = threadIdx.x, sub = tid & 7;
    const int p = tid % HD;
    const int tg = tid / HD;
    const int half = (2 * p) / HD;
    const int r0 = (2 * p) % HD;
    const float* w = static_cast<const float*>(half ? halves[1].w : halves[0].w);
    const float* w0 = w ? w + (size_t)r0 * d : nullptr;
    const int nsteps = d / kKT;

    float ss[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) ss[r] = 0.0f;
    float acc0[TPT], acc1[TPT];
#pragma unroll
    for (int t = 0; t < TPT; ++t) acc0[t] = acc1[t] = 0.0f;

    for (int s = 0; s < nsteps; ++s) {
      float g[8];
      load8(gamma + (size_t)s * kKT + 8 * sub, g);
#pragma unroll
      for (int r = 0; r < CPT; ++r) {
        float x[8];
        load8(hrow[r] + (size_t)s * kKT, x);
        float* dst = hst + (size_t)((tid >> 3) + (NT / 8) * r) * HLD + 8 * sub;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xe = valid[r] ? x[e] : 0.0f;
          ss[r] = fmaf(xe, xe, ss[r]);
          dst[e] = xe * g[e];
        }
      }
      __syncthreads();
      if (w0) {
#pragma unroll 4
        for (int k4 = 0; k4 < kKT / 4; ++k4) {
          const float4 wa = *reinterpret_cast<const float4*>(w0 + (size_t)s * kKT + 4 * k4);
          const float4 wb = *reinterpret_cast<const float4*>(w0 + d + (size_t)s * kKT + 4 * k4);
#pragma unroll
          for (int t = 0; t < TPT; ++t) {
            const float4 hv = *reinterpret_cast<const float4*>(hst + (size_t)(tg * TPT + t) * HLD + 4 * k4);
            acc0[t] = fmaf(wa.x, hv.x, acc0[t]);
            acc0[t] = fmaf(wa.y, hv.y, acc0[t]);
            acc0[t] = fmaf(wa.z, hv.z, acc0[t]);
            acc0[t] = fmaf(wa.w, hv.w, acc0[t]);
            acc1[t] = fmaf(wb.x, hv.x, acc1[t]);
            acc1[t] = fmaf(wb.y, hv.y, acc1[t]);
            acc1[t] = fmaf(wb.z, hv.z, acc1[t]);
            acc1[t] = fmaf(wb.w, hv.w, acc1[t]);
          }
        }
      }
      __syncthreads();
    }

    finish_rms<NT, CPT>(ss, valid, d, eps, rinv);
    __syncthreads();

#pragma unroll
    for (int t = 0; t < TPT; ++t) {
      const int tok = tg * TPT + t;
      const float ri = rinv[tok];
      float v0 = acc0[t] * ri, v1 = acc1[t] * ri;
      if (half ? halves[1].rope : halves[0].rope) rope_rotate(v0, v1, pos[tok], rev[r0 >> 1]);
      *reinterpret_cast<float2*>(kv + (size_t)tok * KLD + half * HD + r0) = make_float2(v0, v1);
    }
  }
};

// ------------------------------------------------------------------ attention

// q heads j*g .. j*g+g-1 of sequence b into LDS: fp32 pre-multiplied by
// log2(e)/sqrt(head_dim), or for bf16 the rows as they are (the MFMA tile
// attention scales its fp32 scores instead).
template <typename T, int HD, int NT>
__device__ __forceinline__ void load_q(const T* q, int b, int n_q, int j, int g, float* qs) {
  constexpr int CH = 16 / sizeof(T);
  const T* src = q + ((size_t)b * n_q + (size_t)j * g) * HD;
  for (int c = threadIdx.x; c < g * HD / CH; c += NT) {
    if constexpr (CH == 8) {
      *reinterpret_cast<u32x4_t*>(reinterpret_cast<uint16_t*>(qs) + CH * c) =
          *reinterpret_cast<const u32x4_t*>(src + CH * c);
    } else {
      const float4 v = *reinterpret_cast<const float4*>(src + CH * c);
      qs[CH * c + 0] = v.x * ScoreScale<HD>::v;
      qs[CH * c + 1] = v.y * ScoreScale<HD>::v;
      qs[CH * c + 2] = v.z * ScoreScale<HD>::v;
      qs[CH * c + 3] = v.w * ScoreScale<HD>::v;
    }
  }
}

// Setup values of a recomputed tile: the KV group's query rows (WITH_Q; as load_q
// stores them), gamma (bf16 with GAMMA, i.e. weights without gamma folded in:
// the fp32 engine reads it from global memory) and the RoPE inverse frequencies.  The constructor issues the loads of a thread's
// first chunks into registers with clamped indexes, unconditionally; store()
// writes the in-range ones to LDS and copies what is left over (more than one q
// chunk or two gamma chunks per thread) with plain loops.  Constructed before a
// tile engine's first loads, stored by its setup(): the two latencies overlap.
template <typename T, int HD, int NT, bool WITH_Q, bool GAMMA = true>
struct TileSetup {
  static constexpr int CH = 16 / sizeof(T);
  const T* qsrc;
  const uint16_t* gsrc;
  int nqc, ngc;
  u32x4_t qv, gv0, gv1;
  double rv;

  __device__ __forceinline__ TileSetup(const T* q, int b, int n_q, int j, int g, const void* gamma, int d,
                                       const double* rev) {
    const int tid = threadIdx.x;
    if constexpr (WITH_Q) {
      qsrc = q + ((size_t)b * n_q + (size_t)j * g) * HD;
      nqc = g * HD / CH;
      qv = *reinterpret_cast<const u32x4_t*>(qsrc + CH * min(tid, nqc - 1));
    }
    rv = rev[min(tid, HD / 2 - 1)];
    if constexpr (sizeof(T) == 2 && GAMMA) {
      gsrc = static_cast<const uint16_t*>(gamma);
      ngc = d / 8;
      gv0 = *reinterpret_cast<const u32x4_t*>(gsrc + 8 * min(tid, ngc - 1));
      gv1 = *reinterpret_cast<const u32x4_t*>(gsrc + 8 * min(tid + NT, ngc - 1));
    }
  }

  __device__ __forceinline__ void store(float* qs, uint16_t* gam, double* revs) const {
    const int tid = threadIdx.x;
    auto put_q = [&](int c, u32x4_t v) {
      float* dst = qs + CH * c;
      if constexpr (CH == 8) {
        *reinterpret_cast<u32x4_t*>(reinterpret_cast<uint16_t*>(qs) + CH * c) = v;
      } else {
        dst[0] = __uint_as_float(v.x) * ScoreScale<HD>::v;
        dst[1] = __uint_as_float(v.y) * ScoreScale<HD>::v;
        dst[2] = __uint_as_float(v.z) * ScoreScale<HD>::v;
        dst[3] = __uint_as_float(v.w) * ScoreScale<HD>::v;
      }
    };
    if constexpr (WITH_Q) {
      if (tid < nqc) put_q(tid, qv);
      for (int c = tid + NT; c < nqc; c += NT) put_q(c, *reinterpret_cast<const u32x4_t*>(qsrc + CH * c));
    }
    if (tid < HD / 2) revs[tid] = rv;
    if constexpr (sizeof(T) == 2 && GAMMA) {
      if (tid < ngc) *reinterpret_cast<u32x4_t*>(gam + 8 * tid) = gv0;
      if (tid + NT < ngc) *reinterpret_cast<u32x4_t*>(gam + 8 * (tid + NT)) = gv1;
      for (int c = tid + 2 * NT; c < ngc; c += NT)
        *reinterpret_cast<uint4*>(gam + 8 * c) = *reinterpret_cast<const uint4*>(gsrc + 8 * c);
    }
  }
};

// Rows row0 .. row0+n-1 (n <= kTile) of a stored K/V block ([B][n_kv][t_cap][HD],
// head j of sequence b) into the LDS tile [kTile][K | V].  Rows wrap around the
// t_cap slots (row0 + t >= t_cap reads slot row0 + t - t_cap; callers keep
// row0 + n <= 2 t_cap): a ring of slots reads oldest first.  All loads of a
// thread are issued before its LDS stores.
template <typename T, int HD, int NT>
__device__ __forceinline__ void load_kv_tile(const T* K, const T* V, int b, int n_kv, int j, int t_cap, int row0,
                                             int n, T* kv) {
  constexpr int KLD = kv_ld<T>(HD);
  constexpr int CH = 16 / sizeof(T);         // elements per 16-byte chunk
  constexpr int CPR = HD / CH;               // chunks per K (or V) row
  constexpr int HALF = kTile * CPR / NT;     // chunks per thread for the K (or V) half of a full tile
  static_assert(HALF * NT == kTile * CPR, "tile split");
  const size_t base = ((size_t)b * n_kv + j) * t_cap;
  u32x4_t v[2 * HALF];
#pragma unroll
  for (int i = 0; i < 2 * HALF; ++i) {
    const int rem = threadIdx.x + NT * (i % HALF);
    const int t = rem / CPR, ch = rem % CPR;
    int row = row0 + (t < n ? t : 0);
    row -= row >= t_cap ? t_cap : 0;
    const T* src = (i < HALF ? K : V) + (base + row) * HD + ch * CH;
    v[i] = *reinterpret_cast<const u32x4_t*>(src);
  }
#pragma unroll
  for (int i = 0; i < 2 * HALF; ++i) {
    const int rem = threadIdx.x + NT * (i % HALF);
    const int t = rem / CPR, ch = rem % CPR;
    if (t < n) *reinterpret_cast<u32x4_t*>(kv + (size_t)t * KLD + (i < HALF ? 0 : HD) + ch * CH) = v[i];
  }
}

// E consecutive elements of a K/V row as floats (E = head_dim / 64).
template <int E> __device__ __forceinline__ void load_e(const uint16_t* p, float (&x)[E]) {
  if constexpr (E == 4) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    x[0] = bf_lo(v.x); x[1] = bf_hi(v.x); x[2] = bf_lo(v.y); x[3] = bf_hi(v.y);
  } else if constexpr (E == 2) {
    const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
    x[0] = bf_lo(v); x[1] = bf_hi(v);
  } else {
    x[0] = to_f<uint16_t>(*p);
  }
}
template <int E> __device__ __forceinline__ void load_e(const float* p, float (&x)[E]) {
#pragma unroll
  for (int e = 0; e < E; ++e) x[e] = p[e];
}

// Stored K/V rows row0 .. row0 + n - 1 (n <= NT / 64) of (b, KV head j) copied
// straight into LDS rows 0 .. n - 1 of `dst` (the K|V row layout of the
// attention tile) by global-to-LDS loads: one wave per row, 16 bytes per lane,
// no registers held, so the copy overlaps whatever the workgroup does next.
// The issuing waves wait for their vector memory counter and the workgroup
// synchronises before the rows are read.
template <typename T, int HD>
__device__ __forceinline__ void prefetch_rows_lds(const T* K, const T* V, size_t row0, int n, T* dst) {
  constexpr int KLD = kv_ld<T>(HD);
  constexpr int CH = 16 / sizeof(T);
  constexpr int CPR = HD / CH;  // 16-byte chunks of a K (or V) row
  const int w = wave_id(), lane = threadIdx.x & 63;
  if (w >= n) return;
#pragma unroll
  for (int c0 = 0; c0 < 2 * CPR; c0 += 64) {
    const int ch = c0 + lane;
    if (ch < 2 * CPR) {
      const T* src = ch < CPR ? K + (row0 + w) * HD + ch * CH : V + (row0 + w) * HD + (ch - CPR) * CH;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                       (__attribute__((address_space(3))) void*)(dst + (size_t)w * KLD + c0 * CH),
                                       16, 0, 0);
    }
  }
}

// Moves n <= kMax K|V rows of the LDS tile from row `from` to row `to` (the
// ranges may overlap): everything is read before anything is written.
// W / LD: elements per row and row stride (the K|V tile by default; one half's
// W = HD, LD = split_ld(HD) on the split engine).
template <typename T, int HD, int NT, int kMax, int W = 2 * HD, int LD = kv_ld<T>(HD)>
__device__ __forceinline__ void move_rows(T* kv, int from, int to, int n) {
  constexpr int KLD = LD;
  constexpr int CH = 16 / sizeof(T);
  constexpr int CPR2 = W / CH;  // 16-byte chunks of a row
  static_assert(kMax * CPR2 <= NT, "one chunk per thread");
  const int r = threadIdx.x / CPR2, ch = threadIdx.x - r * CPR2;
  uint4 v{};
  if (r < n) v = *reinterpret_cast<const uint4*>(kv + (size_t)(from + r) * KLD + ch * CH);
  __syncthreads();
  if (r < n) *reinterpret_cast<uint4*>(kv + (size_t)(to + r) * KLD + ch * CH) = v;
  __syncthreads();
}

// Softmax partial state of one tile of up to 64 * KPL keys (rows of `kv`: K in
// columns [0, HD), V in [HD, 2 HD)) for the g query heads of one KV head, from
// the pre-scaled q in LDS: ml = (max, sum of exp2) per head, and in `red` the
// attn_ts(g) key splits' sums of exp2(s - max) V, whose sum in split order
// (added by write_partial) is the tile's output (Eqs. attn_weights /
// head_output, restricted to the tile).
// Work is split into wave-level tasks whose count depends on g and head_dim
// only, never on the thread count, so every kernel that attends a tile performs
// the same additions in the same order.
//  1. partial scores: task (head h, 64-dim part p), lane = key (and key + 64);
//  2. per head: parts summed in order, max, exp2, sum (one wave per head);
//  3. P V: task (head h, key split ts of attn_ts(g)), lane = head_dim / 64
//     consecutive output columns.
// For n <= 64 the second key slot adds exact zeros (max with -inf, sum with
// 0), so KPL = 1 and KPL = 2 give bit-identical results.  rows >= n is the
// stride of the probabilities in LDS.
// attend_scores runs tasks 1 and 2 (K rows at kt, row stride LD), attend_pv
// task 3 (V rows at vt); attend_tile is the two on one K|V tile.  The split
// engine's K and V roles run one each on their halves, with the probabilities
// and (max, sum) passed between them, and perform the same arithmetic.
template <typename T, int HD, int NT, int KPL, int LD = kv_ld<T>(HD)>
__device__ __forceinline__ void attend_scores(const T* kt, int n, int rows, int g, char* lds, const AttnLds& L) {
  constexpr int KLD = LD;
  constexpr int NW = NT / 64;
  constexpr int P = HD / 64;  // 64-dim parts of a score
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = wave_id();
  const float* qs = reinterpret_cast<const float*>(lds + L.q);
  float* S = reinterpret_cast<float*>(lds + L.s);
  float* red = reinterpret_cast<float*>(lds + L.red);
  float* ml = reinterpret_cast<float*>(lds + L.ml);
  const T* kv = kt;

  static_assert(KPL >= 1 && KPL <= 3, "keys per lane");
  for (int kk = 0; kk < KPL && 64 * kk < n; ++kk) {  // key slot: keys 64 kk + lane
    for (int task = wave; task < g * P; task += NW) {
      const int h = task / P, p = task - h * P;
      const int key = 64 * kk + lane;
      float s = 0.0f;
      if (key < n) {
        const T* krow = kv + (size_t)key * KLD + 64 * p;
        const float* qh = qs + h * HD + 64 * p;
        float d[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          float k8[8];
          load8(krow + 8 * c, k8);
          const float4 qa = *reinterpret_cast<const float4*>(qh + 8 * c);
          const float4 qb = *reinterpret_cast<const float4*>(qh + 8 * c + 4);
          float x = d[c & 3];
          x = fmaf(qa.x, k8[0], x);
          x = fmaf(qa.y, k8[1], x);
          x = fmaf(qa.z, k8[2], x);
          x = fmaf(qa.w, k8[3], x);
          x = fmaf(qb.x, k8[4], x);
          x = fmaf(qb.y, k8[5], x);
          x = fmaf(qb.z, k8[6], x);
          x = fmaf(qb.w, k8[7], x);
          d[c & 3] = x;
        }
        s = (d[0] + d[1]) + (d[2] + d[3]);
      }
      red[(kk * g * P + task) * 64 + lane] = s;
    }
  }
  __syncthreads();

  for (int h = wave; h < g; h += NW) {
    float sk[KPL], pk[KPL];
#pragma unroll
    for (int kk = 0; kk < KPL; ++kk) {
      const float* r = red + (size_t)(kk * g * P + h * P) * 64 + lane;
      sk[kk] = -INFINITY;
      if (64 * kk + lane < n) {
        sk[kk] = r[0];
#pragma unroll
        for (int p = 1; p < P; ++p) sk[kk] += r[64 * p];
      }
    }
    float mx = sk[0];
#pragma unroll
    for (int kk = 1; kk < KPL; ++kk) mx = fmaxf(mx, sk[kk]);
    const float m = wave_max(mx);
#pragma unroll
    for (int kk = 0; kk < KPL; ++kk) pk[kk] = 64 * kk + lane < n ? exp2f(sk[kk] - m) : 0.0f;
    float ps = pk[0];
#pragma unroll
    for (int kk = 1; kk < KPL; ++kk) ps += pk[kk];
    const float l = wave_sum(ps);
#pragma unroll
    for (int kk = 0; kk < KPL; ++kk)
      if (64 * kk + lane < rows) S[h * rows + 64 * kk + lane] = pk[kk];
    if (lane == 0) {
      ml[2 * h] = m;
      ml[2 * h + 1] = l;
    }
  }
  __syncthreads();
}

template <typename T, int HD, int NT, int LD = kv_ld<T>(HD)>
__device__ __forceinline__ void attend_pv(const T* vt, int n, int rows, int g, char* lds, const AttnLds& L) {
  constexpr int KLD = LD;
  constexpr int NW = NT / 64;
  constexpr int E = HD / 64;  // output columns per lane
  const int lane = threadIdx.x & 63;
  const int wave = wave_id();
  const float* S = reinterpret_cast<const float*>(lds + L.s);
  float* red = reinterpret_cast<float*>(lds + L.red);
  const T* kv = vt;
  const int TS = attn_ts(g);
  for (int task = wave; task < g * TS; task += NW) {
    const int h = task % g, ts = task / g;
    float a[E];
#pragma unroll
    for (int e = 0; e < E; ++e) a[e] = 0.0f;
    int t = ts;
    for (; t + 3 * TS < n; t += 4 * TS) {  // four keys' reads in flight, then their sums in key order
      float pr[4], v[4][E];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        pr[k] = S[h * rows + t + k * TS];
        load_e<E>(kv + (size_t)(t + k * TS) * KLD + E * lane, v[k]);
      }
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int e = 0; e < E; ++e) a[e] = fmaf(pr[k], v[k][e], a[e]);
    }
    for (; t < n; t += TS) {
      const float pr = S[h * rows + t];
      float v[E];
      load_e<E>(kv + (size_t)t * KLD + E * lane, v);
#pragma unroll
      for (int e = 0; e < E; ++e) a[e] = fmaf(pr, v[e], a[e]);
    }
    float* dst = red + ((size_t)ts * g + h) * HD + E * lane;
#pragma unroll
    for (int e = 0; e < E; ++e) dst[e] = a[e];
  }
  __syncthreads();
}

// The bf16 tile attention on 16x16x32 MFMAs, in the same two halves and with
// the same results in LDS: probabilities S[h * rows + key] and (max, sum) per
// head from attend_scores_mfma, the tile's P V per head in `red` from
// attend_pv_mfma (write_partial then takes one key split).  q sits in LDS as raw
// bf16 rows.
//  1. scores: task (16-key block, group of 16 heads): S^T = K q^T over HD / 32
//     k-steps, A = 16 key rows of the tile, B = the heads' q rows; a lane gets
//     4 keys of one head, scaled by log2(e)/sqrt(head_dim) in fp32;
//  2. per head (one wave each): max, p = 2^(s - max) rounded to bf16 (the value
//     the P V product uses), sum of the rounded p;
//  3. P V: task (16 output columns, group of 16 heads): O^T = V^T P^T over
//     32-key steps in key order, A = V^T fetched from the row-major V rows by
//     two LDS transpose reads (4 keys of one column each), B = the heads'
//     probabilities.
// Keys past n contribute zeros: their probabilities are 0 and their V^T
// elements are replaced by 0 before the product (LDS past the tile may hold
// anything).  Rows past the tile are clamped to its last row for the reads.
// Row strides of S (rows) and of the K|V tile keep every 16-byte read aligned
// (rows and LD multiples of 4 and 8 elements).
template <int HD, int NT, int KPL, int LD = kv_ld<uint16_t>(HD)>
__device__ __forceinline__ void attend_scores_mfma(const uint16_t* kt, int n, int rows, int g, char* lds,
                                                   const AttnLds& L) {
  constexpr int NW = NT / 64;
  constexpr int SR = 64 * KPL;  // row stride of the raw scores in `red`
  static_assert(KPL >= 1 && KPL <= 3 && HD % 32 == 0, "keys per lane, k-steps");
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int lq = lane & 15, lg = lane >> 4;
  const uint16_t* qb = reinterpret_cast<const uint16_t*>(lds + L.q);
  float* sc = reinterpret_cast<float*>(lds + L.red);
  float* S = reinterpret_cast<float*>(lds + L.s);
  float* ml = reinterpret_cast<float*>(lds + L.ml);
  const int nkb = (n + 15) >> 4, nhg = (g + 15) >> 4;
  for (int task = wave; task < nkb * nhg; task += NW) {
    const int kb = task % nkb, hgp = task / nkb;
    const int head = 16 * hgp + lq;
    const uint16_t* ka = kt + (size_t)min(16 * kb + lq, rows - 1) * LD + 8 * lg;
    const uint16_t* qa = qb + (size_t)min(head, g - 1) * HD + 8 * lg;
    f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ks = 0; ks < HD / 32; ++ks)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*reinterpret_cast<const bf16x8_t*>(ka + 32 * ks),
                                                    *reinterpret_cast<const bf16x8_t*>(qa + 32 * ks), acc, 0, 0, 0);
    if (head < g)
      *reinterpret_cast<float4*>(sc + (size_t)head * SR + 16 * kb + 4 * lg) =
          make_float4(acc[0] * ScoreScale<HD>::v, acc[1] * ScoreScale<HD>::v, acc[2] * ScoreScale<HD>::v,
                      acc[3] * ScoreScale<HD>::v);
  }
  __syncthreads();

  for (int h = wave; h < g; h += NW) {
    float sk[KPL], pk[KPL];
#pragma unroll
    for (int kk = 0; kk < KPL; ++kk) {
      const int key = 64 * kk + lane;
      sk[kk] = key < n ? sc[(size_t)h * SR + key] : -INFINITY;
    }
    float mx = sk[0];
#pragma unroll
    for (int kk = 1; kk < KPL; ++kk) mx = fmaxf(mx, sk[kk]);
    const float m = wave_max(mx);
#pragma unroll
    for (int kk = 0; kk < KPL; ++kk) pk[kk] = 64 * kk + lane < n ? bf_lo(pack_bf16x2(exp2f(sk[kk] - m), 0.0f)) : 0.0f;
    float ps = pk[0];
#pragma unroll
    for (int kk = 1; kk < KPL; ++kk) ps += pk[kk];
    const float l = wave_sum(ps);
#pragma unroll
    for (int kk = 0; kk < KPL; ++kk)
      if (64 * kk + lane < rows) S[h * rows + 64 * kk + lane] = pk[kk];
    if (lane == 0) {
      ml[2 * h] = m;
      ml[2 * h + 1] = l;
    }
  }
  __syncthreads();
}

template <int HD, int NT, int LD = kv_ld<uint16_t>(HD)>
__device__ __forceinline__ void attend_pv_mfma(const uint16_t* vt, int n, int rows, int g, char* lds,
                                               const AttnLds& L) {
  typedef short i16x4_t __attribute__((ext_vector_type(4)));
  constexpr int NW = NT / 64;
  constexpr int NDB = HD / 16;  // 16-column blocks of the output
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int lq = lane & 15, lg = lane >> 4;
  const float* S = reinterpret_cast<const float*>(lds + L.s);
  float* red = reinterpret_cast<float*>(lds + L.red);
  const int nks = (n + 31) >> 5, nhg = (g + 15) >> 4;
  // transpose reads: within each group of 16 lanes, lane s reads 4 columns
  // 4 (s % 4) .. of row s / 4 of a 4-row group; lane i then holds column i of
  // the group's 4 rows
  const int sr = lq >> 2, scol = 4 * (lq & 3);
  for (int task = wave; task < NDB * nhg; task += NW) {
    const int db = task % NDB, hgp = task / NDB;
    const int head = 16 * hgp + lq;
    const float* prow = S + (size_t)min(head, g - 1) * rows;
    const uint16_t* vcol = vt + 16 * db + scol;
    f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int ks = 0; ks < nks; ++ks) {
      const int k0 = 32 * ks + 8 * lg;  // keys k0 .. k0 + 7 of this lane (both operands)
      i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) i16x4_t*)(vcol + (size_t)min(k0 + sr, rows - 1) * LD));
      i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) i16x4_t*)(vcol + (size_t)min(k0 + 4 + sr, rows - 1) * LD));
      const float4 p0 = *reinterpret_cast<const float4*>(prow + k0);
      const float4 p1 = *reinterpret_cast<const float4*>(prow + k0 + 4);
      float pv[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
      if (k0 + 8 > n) {  // the keys past n: zero weights and zero values
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (k0 + e >= n) {
            lo[e] = 0;
            pv[e] = 0.0f;
          }
          if (k0 + 4 + e >= n) {
            hi[e] = 0;
            pv[4 + e] = 0.0f;
          }
        }
      }
      const bf16x8_t a = __builtin_bit_cast(
          bf16x8_t, make_uint4(__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                               __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y));
      const bf16x8_t bp = __builtin_bit_cast(bf16x8_t, make_uint4(pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                                                                  pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])));
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bp, acc, 0, 0, 0);
    }
    if (head < g)
      *reinterpret_cast<float4*>(red + (size_t)head * HD + 16 * db + 4 * lg) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  }
  __syncthreads();
}

// Key splits of the P V partial sums a tile's attention leaves in `red`.
template <typename T>
__device__ __forceinline__ int tile_splits(int g) {
  return sizeof(T) == 2 ? 1 : attn_ts(g);
}

template <typename T, int HD, int NT, int KPL>
__device__ __forceinline__ void attend_tile(const T* kv, int n, int rows, int g, char* lds, const AttnLds& L) {
  if constexpr (sizeof(T) == 2) {
    attend_scores_mfma<HD, NT, KPL>(kv, n, rows, g, lds, L);
    attend_pv_mfma<HD, NT>(kv + HD, n, rows, g, lds, L);
  } else {
    attend_scores<T, HD, NT, KPL>(kv, n, rows, g, lds, L);
    attend_pv<T, HD, NT>(kv + HD, n, rows, g, lds, L);
  }
}

// Device-scope (coherent across the XCDs' L2 caches) 32-bit store / load: the
// split-K partials cross workgroups on different XCDs, so they are written
// through and read past the per-XCD L2 instead of fencing whole caches.
__device__ __forceinline__ void store_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Split-K partial of (b, KV head j, split s) into the workspace:
// acc [B][n_q][S][HD] fp32 followed by ml [B][n_q][S][2] fp32.  The tile's
// output is the sum, in key-split order, of the TS P V partial sums the tile
// attention left in `red` (tile_splits); it is added here as it is written out.
template <int HD, int NT>
__device__ __forceinline__ void write_partial(const char* lds, const AttnLds& L, float* ws_acc, float* ws_ml, int b,
                                              int n_q, int j, int g, int S, int s, int TS) {
  const float* red = reinterpret_cast<const float*>(lds + L.red);
  const float* ml = reinterpret_cast<const float*>(lds + L.ml);
  for (int i = threadIdx.x; i < g * HD; i += NT) {
    const int h = i / HD, c = i - h * HD;
    float o = 0.0f;
    for (int ts = 0; ts < TS; ++ts) o += red[(size_t)ts * g * HD + i];
    store_dev(ws_acc + (((size_t)b * n_q + (size_t)j * g + h) * S + s) * HD + c, o);
  }
  if (threadIdx.x < 2 * g) {
    const int h = threadIdx.x >> 1;
    store_dev(ws_ml + (((size_t)b * n_q + (size_t)j * g + h) * S + s) * 2 + (threadIdx.x & 1), ml[threadIdx.x]);
  }
}

// Merge of the S split-K partial states of rows row0 .. row0+nrows-1 (row =
// b * n_q + query head) into out (Eqs. attn_weights / head_output over all
// splits): M = max_s m_s, w_s = 2^(m_s - M), out = sum_s w_s acc_s / sum_s w_s l_s.
// Every sum has a fixed order that does not depend on NT: each output column
// adds its splits in split order; the denominator is accumulated per lane over
// splits s = lane, lane + 64, ... and then summed by the fixed wave tree.  A
// pass merges RPP rows: each thread owns one column of CPT of them (CPT = 2
// for head_dim >= 128), so a decode group's rows go in one pass; splits go in
// blocks of 64.  The (max, sum) pairs of the first kCmbKeep blocks are loaded
// once and kept in registers, and every thread issues all of a block's
// accumulator loads (partial blocks included) before its first wait, while the
// waves that own the rows' weights compute them: one round trip per block.
// CPT2 asks for two columns per thread where the rows allow it (64 more
// registers of accumulators in flight); the arithmetic is the same either way.
// lds: cmb_floats(NT, HD) floats.
template <typename T, int HD, int NT, bool CPT2 = false>
__device__ __forceinline__ void combine_rows(const float* ws_acc, const float* ws_ml, T* out, size_t row0, int nrows,
                                             int S, float* lds) {
  constexpr int RPH = NT / HD;                                  // rows per column set (one column per thread)
  constexpr int CPT = CPT2 && 2 * RPH <= NT / 64 ? 2 : 1;      // columns per thread
  constexpr int RPP = CPT * RPH;                                // rows per pass
  constexpr int KEEP = kCmbKeep;
  static_assert(RPH >= 1 && RPP <= NT / 64 && RPP * 66 <= (int)cmb_floats(NT, HD), "rows per pass");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = wave_id();
  const int rr = tid / HD, c = tid - rr * HD;
  float* wsh = lds;             // [RPP][64] weights of the current block of splits
  float* mL = lds + RPP * 64;   // [RPP][2] max, denominator
  for (int r0 = 0; r0 < nrows; r0 += RPP) {
    const bool mine = wave < RPP && r0 + wave < nrows;  // this wave owns the weights of row r0 + wave
    bool rv[CPT];                                         // this thread owns column c of row r0 + rr + k RPH
#pragma unroll
    for (int k = 0; k < CPT; ++k) rv[k] = rr < RPH && r0 + rr + k * RPH < nrows;
    const float* mlw = ws_ml + (row0 + r0 + wave) * (size_t)S * 2;
    // accumulators: a uniform base per block plus a 32-bit per-lane offset
    const float* abase = ws_acc + (row0 + r0) * (size_t)S * HD;
    unsigned aoff[CPT];
#pragma unroll
    for (int k = 0; k < CPT; ++k) aoff[k] = (unsigned)((rr + k * RPH) * S * HD + c);
    float mv[KEEP], lv[KEEP];
    float M = -INFINITY;
    if (mine) {
#pragma unroll
      for (int k = 0; k < KEEP; ++k) {
        const int s = 64 * k + lane;
        mv[k] = s < S ? load_dev(mlw + 2 * s) : -INFINITY;
        lv[k] = s < S ? load_dev(mlw + 2 * s + 1) : 0.0f;
      }
    }
    float o[CPT], lsum = 0.0f;
#pragma unroll
    for (int k = 0; k < CPT; ++k) o[k] = 0.0f;
    for (int s0 = 0, blk = 0; s0 < S; s0 += 64, ++blk) {
      const int cnt = min(64, S - s0);
      const float* a = abase + (size_t)s0 * HD;
      // the block's accumulators: every load in flight before any wait, in chunks
      // of 8 splits (a uniform branch per chunk; within the last chunk, loads past
      // the last split repeat split cnt - 1: in bounds and finite, weight zero)
      float x[CPT][64];
#pragma unroll
      for (int k = 0; k < CPT; ++k) {
        if (rv[k]) {
#pragma unroll
          for (int e0 = 0; e0 < 64; e0 += 8) {
            if (e0 < cnt) {
#pragma unroll
              for (int e = e0; e < e0 + 8; ++e) x[k][e] = load_dev(a + (size_t)min(e, cnt - 1) * HD + aoff[k]);
            }
          }
        }
      }
      if (mine) {
        if (blk == 0) {  // the maximum over all splits, before the first weight
          float m = mv[0];
#pragma unroll
          for (int k = 1; k < KEEP; ++k) m = fmaxf(m, mv[k]);
          for (int s = 64 * KEEP + lane; s < S; s += 64) m = fmaxf(m, load_dev(mlw + 2 * s));
          M = wave_max(m);
        }
        const int s = s0 + lane;
        float mk = -INFINITY, lk = 0.0f;
#pragma unroll
        for (int k = 0; k < KEEP; ++k)
          if (blk == k) mk = mv[k], lk = lv[k];
        if (blk >= KEEP && s < S) mk = load_dev(mlw + 2 * s), lk = load_dev(mlw + 2 * s + 1);
        const float w = s < S ? exp2f(mk - M) : 0.0f;
        lsum = fmaf(lk, w, lsum);
        wsh[wave * 64 + lane] = w;
      }
      __syncthreads();
      // chunks past the last split are skipped; inside the last chunk w = 0 past
      // the last split, so those terms add an exact zero
#pragma unroll
      for (int k = 0; k < CPT; ++k) {
        if (rv[k]) {
          const float* wp = wsh + (rr + k * RPH) * 64;
#pragma unroll
          for (int e0 = 0; e0 < 64; e0 += 8) {
            if (e0 < cnt) {
#pragma unroll
              for (int e = e0; e < e0 + 8; ++e) o[k] = fmaf(x[k][e], wp[e], o[k]);
            }
          }
        }
      }
      __syncthreads();
    }
    if (mine) {
      lsum = wave_sum(lsum);
      if (lane == 0) mL[2 * wave + 1] = lsum;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < CPT; ++k)
      if (rv[k]) out[(row0 + r0 + rr + k * RPH) * HD + c] = from_f<T>(o[k] / mL[2 * (rr + k * RPH) + 1]);
    __syncthreads();
  }
}

// Split-K completion counter of (b, KV head j): one 64-bit word in the
// workspace whose low 32 bits count the splits whose partials are written (the
// high 32 bits are reserved and stay zero).  Every thread first waits for its own
// device-scope partial stores to complete; then one thread adds `add` and the
// value before the add is broadcast to the workgroup.
// No cache-wide write-back or invalidate is needed, so other workgroups that
// stream weights through the same L2 keep them.
__device__ __forceinline__ unsigned long long split_arrive(unsigned long long* ctr, unsigned long long add,
                                                           unsigned long long* bcast) {
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  __syncthreads();
  if (threadIdx.x == 0) *bcast = __hip_atomic_fetch_add(ctr, add, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  return *bcast;
}

// True in the one workgroup whose add of `added` completed splits brought the
// count to S: every partial is then written, and reads with load_dev see them.
// That workgroup resets the word for the next call (no add can follow: all S
// splits, hence all arrivals, are counted).
__device__ __forceinline__ bool split_complete(unsigned long long* ctr, unsigned long long before, unsigned added,
                                               int S) {
  const bool last = (unsigned)(before & 0xffffffffull) + added == (unsigned)S;
  if (last && threadIdx.x == 0) __hip_atomic_store(ctr, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return last;
}

}  // namespace kvd
