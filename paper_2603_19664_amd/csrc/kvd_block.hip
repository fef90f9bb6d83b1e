// Kernels of the single-checkpoint scheme: one pre-norm transformer block over
// all positions (Sec. 3.1, Eqs. q_proj .. mlp_sublayer), run layer after layer
// to recompute h^(l) from the one stored residual per token (Eq. res_mem).
// The Q/K/V projections are the recompute tile engine's (proj_kernel); this file
// holds the output projections (W_o, and the MLP's gate/up and down) on the same
// MFMA tile engine with other epilogues, and causal prefill attention.
#include <hip/hip_runtime.h>

#include <atomic>

#include <algorithm>

#include "kvd_device.hpp"
#include "kvd_launch.h"

namespace kvd {

// ------------------------------------------------------------------ projections with residual / SwiGLU epilogues

// grid: xcd_map(n_units * n_tiles) workgroups; item = unit * n_tiles + tile (the
// token tiles of one weight block run on one XCD).  A unit is 512 rows of W
// (kEpiResidual) or 256 rows each of W and W2 (kEpiSwiglu); a tile is MT token
// rows: 64 on MfmaTile, or 128 on WideTile for launches with at least a full
// round of such tiles.  Both engines give wave w rows 32 w .. 32 w + 31 of each
// half and run the same per-element MFMA chain, so the outputs are identical.
template <int EPI, bool NORM, bool PACKED, int MT>
__global__ __launch_bounds__(kNtTile, 1) void gemm_kernel(GemmArgs a, int per_xcd, int n_tiles, int n_units) {
  extern __shared__ __align__(16) char lds[];
  constexpr int NT = kNtTile, HD = 256;
  constexpr ProjLds PL = proj_lds<uint16_t>(HD, MT);
  constexpr int KLD = kv_ld<uint16_t>(HD);
  using Tile = MfmaTile<HD, kMtBf16, PACKED>;
  using Wide = WideTile<HD, 2 * kMtBf16, PACKED, false, kNtWide, kv_ld<uint16_t>(HD), false, true>;
  static_assert(MT == kMtBf16 || MT == 2 * kMtBf16, "64- or 128-token tiles");
  static_assert(Tile::NB_F == 2 && Tile::WT == 1 && Tile::NB_T == 2 && Wide::NB_F == 2 && NT == Wide::NT,
                "wave w owns rows 32 w.. of both halves");
  const int tid = threadIdx.x;
  // 32-bit index arithmetic: the launch's grid bounds the item count
  const unsigned item = (blockIdx.x % kXcds) * (unsigned)per_xcd + blockIdx.x / kXcds;
  if (item >= (unsigned)n_units * (unsigned)n_tiles) return;
  const int unit = (int)(item / (unsigned)n_tiles);
  const int tile = (int)(item - (unsigned)unit * (unsigned)n_tiles);
  float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
  uint16_t* hst = reinterpret_cast<uint16_t*>(lds + PL.hst);
  uint16_t* kv = reinterpret_cast<uint16_t*>(lds + PL.kv);
  uint16_t* gam = reinterpret_cast<uint16_t*>(lds + PL.end);
  const long long n0 = (long long)tile * MT;
  const size_t K = (size_t)a.K;
  const uint16_t* W = static_cast<const uint16_t*>(a.w);
  Half halves[2];
  if constexpr (EPI == kEpiResidual) {
    halves[0] = Half{W + (size_t)512 * unit * K, 0};
    halves[1] = Half{W + ((size_t)512 * unit + 256) * K, 0};
  } else {
    halves[0] = Half{W + (size_t)256 * unit * K, 0};
    halves[1] = Half{static_cast<const uint16_t*>(a.w2) + (size_t)256 * unit * K, 0};
  }
  const uint16_t* hrow[1];
  bool valid[1];
  {
    long long n = n0 + (tid >> 3);
    valid[0] = n < a.M;
    if (!valid[0]) n = n0;  // any readable row; its column is not stored
    hrow[0] = static_cast<const uint16_t*>(a.x) + (size_t)n * K + 8 * (tid & 7);
  }
  const int n_rows = (int)std::min<long long>(MT, a.M - n0);
  // gamma (or ones) into LDS while the K-loop's first loads are in flight
  const uint16_t* gsrc = static_cast<const uint16_t*>(a.gamma);
  const int ngc = a.K / 8;
  const u32x4_t gv0 = *reinterpret_cast<const u32x4_t*>(gsrc + 8 * min(tid, ngc - 1));
  const u32x4_t gv1 = *reinterpret_cast<const u32x4_t*>(gsrc + 8 * min(tid + NT, ngc - 1));
  auto setup = [&]() {
    if (tid < ngc) *reinterpret_cast<u32x4_t*>(gam + 8 * tid) = gv0;
    if (tid + NT < ngc) *reinterpret_cast<u32x4_t*>(gam + 8 * (tid + NT)) = gv1;
    for (int c = tid + 2 * NT; c < ngc; c += NT)
      *reinterpret_cast<u32x4_t*>(gam + 8 * c) = *reinterpret_cast<const u32x4_t*>(gsrc + 8 * c);
  };
  const int lane = tid & 63, fw = wave_id() % Tile::WF;
  auto epi = [&](const auto& acc, const auto&) {
#pragma unroll
                   for (int bt = 0; bt < MT / 32; ++bt) {
                     const int tok = 32 * bt + (lane & 31);
                     const long long n = n0 + tok;
                     const float ri = NORM ? rinv[tok] : 1.0f;
#pragma unroll
                     for (int g4 = 0; g4 < 4; ++g4) {
                       const int f = 32 * fw + 8 * g4 + 4 * (lane >> 5);  // features f .. f+3 of each half
                       if constexpr (EPI == kEpiResidual) {
#pragma unroll
                         for (int bf = 0; bf < 2; ++bf) {
                           float v[4];
#pragma unroll
                           for (int e = 0; e < 4; ++e) v[e] = acc[bf][bt][4 * g4 + e] * ri;
                           if (n < a.M) {
                             const uint2 r = *reinterpret_cast<const uint2*>(
                                 static_cast<const uint16_t*>(a.res) + (size_t)n * a.N + 512 * unit + 256 * bf + f);
                             v[0] += bf_lo(r.x);
                             v[1] += bf_hi(r.x);
                             v[2] += bf_lo(r.y);
                             v[3] += bf_hi(r.y);
                           }
                           uint2 o;
                           o.x = pack_bf16x2(v[0], v[1]);
                           o.y = pack_bf16x2(v[2], v[3]);
                           *reinterpret_cast<uint2*>(kv + (size_t)tok * KLD + 256 * bf + f) = o;
                         }
                       } else {
                         float v[4];
#pragma unroll
                         for (int e = 0; e < 4; ++e) {
                           const float gt = acc[0][bt][4 * g4 + e] * ri, ut = acc[1][bt][4 * g4 + e] * ri;
                           v[e] = gt / (1.0f + expf(-gt)) * ut;
                         }
                         uint2 o;
                         o.x = pack_bf16x2(v[0], v[1]);
                         o.y = pack_bf16x2(v[2], v[3]);
                         *reinterpret_cast<uint2*>(kv + (size_t)tok * KLD + f) = o;
                       }
                     }
                   }
  };
  if constexpr (MT == kMtBf16)
    Tile::run_with(hrow, valid, gam, gsrc, a.K, a.eps, halves, hst, rinv, setup, epi);
  else
    Wide::run_with(static_cast<const uint16_t*>(a.x) + (size_t)n0 * K, n_rows, gam, gsrc, a.K, a.eps, halves, hst,
                   rinv, setup, epi);
  __syncthreads();
  // store: 16-byte chunks of the valid token rows
  constexpr int NF = EPI == kEpiResidual ? 512 : 256;
  const size_t col0 = (size_t)NF * unit;
  uint16_t* out = static_cast<uint16_t*>(a.out);
  for (int c = tid; c < MT * NF / 8; c += NT) {
    const int row = c / (NF / 8), ch = c - row * (NF / 8);
    const long long n = n0 + row;
    if (n >= a.M) continue;
    *reinterpret_cast<uint4*>(out + (size_t)n * a.N + col0 + 8 * ch) =
        *reinterpret_cast<const uint4*>(kv + (size_t)row * KLD + 8 * ch);
  }
}

// ------------------------------------------------------------------ causal prefill attention

// LDS of prefill_attn_kernel (bytes): the workgroup's query rows [128][HD + 8],
// the key tile and the value tile [64][HD + 8], bf16.
struct PrefillLds {
  size_t qs, ks, vs, ctr, end;
};
constexpr PrefillLds prefill_lds(int hd) {
  PrefillLds L{};
  L.qs = 0;
  L.ks = L.qs + (size_t)2 * 128 * (hd + 8);
  L.vs = L.ks + (size_t)2 * 64 * (hd + 8);
  L.ctr = L.vs + (size_t)2 * 64 * (hd + 8);  // split counter broadcast
  L.end = L.ctr + 16;
  return L;
}

// grid: (pieces of one head) * B * n_q workgroups, 256 threads (4 waves), item =
// blockIdx.x.  A piece is a (query block, key part) pair; the host lists them
// longest first (order), and items run (piece rank, sequence, KV head, query head
// of the group), so the longest pieces start first and consecutive items go to
// different XCDs, which gives every XCD its share of each rank.  Without a list
// (too many blocks, then nothing is split) rank r is query block nqb - 1 - r.  A
// workgroup takes 128 query rows of one head, 32 per wave, through the key
// blocks of 64 of its part of the range up to its last row (flash order),
// loading block kb + 1 into registers while block kb is computed.
//
// Scores are computed transposed, S^T = K Q^T: A = 32 keys from the LDS tile,
// B = the wave's 32 query rows (registers), so that a lane holds one query's
// scores in its registers and the softmax needs no LDS: the running max and sum
// of a query live in the two lanes (l, l ^ 32) that hold its keys, and the max
// used for the weights moves only in steps of more than 2^8 (rescaling then).  The output is
// accumulated transposed too, O^T += V^T P^T, with P^T straight from the score
// registers: for the 16 keys of an MFMA step, lane half h supplies the keys its
// score registers hold (32 kh + 16 (t & 1) + 4 h + {0..3, 8..11}), and the V^T
// operand takes the same keys, so both operands agree on the reduction order.
// V stays row-major in LDS; each V^T operand is two LDS transpose reads (in a
// group of 16 lanes, lane s names 4 columns of row s / 4 of a 4-key group, and
// lane i receives column i of the 4 keys).
// Scores are in the log2 domain (log2(e) / sqrt(hd) folded into the scale).
template <int HD>
__global__ __launch_bounds__(256) void prefill_attn_kernel(PrefillArgs a) {
  extern __shared__ __align__(16) char lds[];
  constexpr PrefillLds PL = prefill_lds(HD);
  constexpr int KS = HD / 16;              // 16-wide k-steps of a score block
  constexpr int DB = HD / 32;              // 32-row blocks of O^T (head_dim rows)
  constexpr int KLDS = HD + 8;
  constexpr int CPR = HD / 8;              // 16-byte chunks per key row
  constexpr int KCH = 64 * CPR / 256;      // key (and value) chunks per thread
  typedef short i16x4_t __attribute__((ext_vector_type(4)));
  uint16_t* Qs = reinterpret_cast<uint16_t*>(lds + PL.qs);
  uint16_t* Ks = reinterpret_cast<uint16_t*>(lds + PL.ks);
  uint16_t* Vs = reinterpret_cast<uint16_t*>(lds + PL.vs);

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int hl = lane >> 5;  // lane half
  const int nqb = (a.T + 127) / 128;
  const int g = a.n_q / a.n_kv;
  // 32-bit index arithmetic: the launch's grid bounds the item count
  const unsigned item = blockIdx.x;
  const int hh = (int)(item % (unsigned)g);
  const unsigned r0 = item / (unsigned)g;
  const unsigned bj = (unsigned)a.B * (unsigned)a.n_kv;
  const int j = (int)(r0 % (unsigned)a.n_kv);
  const int b = (int)((r0 / (unsigned)a.n_kv) % (unsigned)a.B);
  const int rank = (int)(r0 / bj);
  const unsigned piece = a.n_order > 0 ? a.order[rank] : (unsigned)(nqb - 1 - rank) << 8;
  const int qb = (int)(piece >> 8), part = (int)(piece & 255u);
  const int h = j * g + hh;
  const int last_row = min(128 * qb + 127, a.T - 1);
  const int nkb = last_row / 64 + 1;        // key blocks 0 .. nkb - 1 reach this block's rows
  const int np = (nkb + a.P - 1) / a.P;     // parts of the key range
  const int kb0 = part * nkb / np, kb1 = (part + 1) * nkb / np;
  const int q0 = 128 * qb + 32 * w;          // this wave's first query row
  const int query = q0 + (lane & 31);        // this lane's query row
  const float scale = ScoreScale<HD>::v;
  const uint16_t* kbase = static_cast<const uint16_t*>(a.k) + ((size_t)b * a.n_kv + j) * a.T * HD;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + ((size_t)b * a.n_kv + j) * a.T * HD;

  // the wave's query rows into LDS (its own 32 rows; read back as MFMA B
  // operands: column = query, 8 dims per lane half)
  for (int c = lane; c < 32 * CPR; c += 64) {
    const int row = c / CPR, ch = c - row * CPR;
    const int t = min(q0 + row, a.T - 1);
    *reinterpret_cast<u32x4_t*>(Qs + (32 * w + row) * KLDS + 8 * ch) = *reinterpret_cast<const u32x4_t*>(
        static_cast<const uint16_t*>(a.q) + (((size_t)b * a.T + t) * a.n_q + h) * HD + 8 * ch);
  }
  const uint16_t* qrow = Qs + (32 * w + (lane & 31)) * KLDS + 8 * hl;
  f32x16_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  // key / value block kb into registers (rows clamped to T - 1: masked below)
  u32x4_t kc[KCH], vc[KCH];
  auto load_kv = [&](int kb) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + 256 * i, row = c / CPR, ch = c - row * CPR;
      const size_t t = min(64 * kb + row, a.T - 1);
      kc[i] = *reinterpret_cast<const u32x4_t*>(kbase + t * HD + 8 * ch);
      vc[i] = *reinterpret_cast<const u32x4_t*>(vbase + t * HD + 8 * ch);
    }
  };
  load_kv(kb0);

  for (int kb = kb0; kb < kb1; ++kb) {
    // the registers into LDS, both row-major
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + 256 * i, row = c / CPR, ch = c - row * CPR;
      *reinterpret_cast<u32x4_t*>(Ks + row * KLDS + 8 * ch) = kc[i];
      *reinterpret_cast<u32x4_t*>(Vs + row * KLDS + 8 * ch) = vc[i];
    }
    __syncthreads();
    if (kb + 1 < kb1) load_kv(kb + 1);  // in flight while this block is computed

    // a wave whose rows all precede the block (or lie past T) skips it
    if (64 * kb <= q0 + 31 && q0 < a.T) {
      // S^T for key halves kh = 0, 1: four independent accumulator chains
      f32x16_t st[2], sx[2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int i = 0; i < 16; ++i) st[kh][i] = sx[kh][i] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ks += 2) {
        const bf16x8_t q0f = *reinterpret_cast<const bf16x8_t*>(qrow + 16 * ks);
        const bf16x8_t q1f = *reinterpret_cast<const bf16x8_t*>(qrow + 16 * ks + 16);
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
          const uint16_t* kr = Ks + (32 * kh + (lane & 31)) * KLDS + 8 * hl + 16 * ks;
          const bf16x8_t k0 = *reinterpret_cast<const bf16x8_t*>(kr);
          const bf16x8_t k1 = *reinterpret_cast<const bf16x8_t*>(kr + 16);
          st[kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, q0f, st[kh], 0, 0, 0);
          sx[kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, q1f, sx[kh], 0, 0, 0);
        }
      }
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 64 * kb + 32 * kh + 8 * (r >> 2) + 4 * hl + (r & 3);
          float v = (st[kh][r] + sx[kh][r]) * scale;
          if (query >= a.T) v = 0.0f;  // rows past the end: finite, never stored
          else if (key > query) v = -INFINITY;
          st[kh][r] = v;
        }
      // running softmax of this lane's query: its 32 scores here and 32 in lane ^ 32
      float mx = -INFINITY;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[kh][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      // The reference max moves only when the block's max exceeds it by more than 8
      // (log2 units): the weights 2^(s - m) stay <= 2^8, and O and l are rescaled
      // (accumulators held in AGPRs) only in the few blocks where it moves.
      const bool grow = mx > m_run + 8.0f;
      if (__any(grow)) {
        const float m_new = grow ? mx : m_run;
        const float alpha = exp2f(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
      }
      bf16x8_t pf[4];  // P^T operands of the four 16-key MFMA steps
      float sum = 0.0f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        uint32_t pw[4];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const int r = 8 * (t & 1) + e;
          pw[e >> 1] = pack_bf16x2(exp2f(st[t >> 1][r] - m_run), exp2f(st[t >> 1][r + 1] - m_run));
          sum += bf_lo(pw[e >> 1]) + bf_hi(pw[e >> 1]);  // the rounded weights the MFMA uses
        }
        pf[t] = __builtin_bit_cast(bf16x8_t, make_uint4(pw[0], pw[1], pw[2], pw[3]));
      }
      sum += __shfl_xor(sum, 32, 64);
      l_run += sum;
      // O^T += V^T P^T: per 16-key step, the DB accumulators are independent.
      // Transpose-read source of this lane: keys k0 + 4 hl + (lane % 16) / 4
      // (+ 8 for the upper four), columns 32 db + 16 ((lane / 16) % 2) +
      // 4 (lane % 4) .. + 3.
      const uint16_t* vsrc = Vs + (4 * hl + ((lane & 15) >> 2)) * KLDS + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int k0 = 32 * (t >> 1) + 16 * (t & 1);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const uint16_t* vr = vsrc + k0 * KLDS + 32 * db;
          const i16x4_t lo =
              __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4_t*)vr);
          const i16x4_t hi =
              __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4_t*)(vr + 8 * KLDS));
          const bf16x8_t vf = __builtin_bit_cast(
              bf16x8_t, make_uint4(__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                                   __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y));
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[t], o[db], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  if (np > 1) {
    // This part's state into its slot (per wave: O as [db][r][lane], then the
    // lane's max and sum), then the arrival; the last part merges every part's
    // state in part order, so the result does not depend on which part arrives
    // last.
    constexpr size_t PF = 4 * (DB * 16 * 64 + 128);
    const size_t blk = ((size_t)b * a.n_q + h) * nqb + qb;
    float* slots = a.part + blk * a.NP * PF;
    {
      float* so = slots + (size_t)part * PF + (size_t)w * DB * 16 * 64 + lane;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) store_dev(so + (db * 16 + r) * 64, o[db][r]);
      float* sm = slots + (size_t)part * PF + 4 * DB * 16 * 64 + w * 128 + lane;
      store_dev(sm, m_run);
      store_dev(sm + 64, l_run);
    }
    unsigned long long* ctr = a.ctr + blk;
    const unsigned long long before =
        split_arrive(ctr, 1, reinterpret_cast<unsigned long long*>(lds + PL.ctr));
    if (!split_complete(ctr, before, 1, np)) return;
    // O = sum over parts p (in order) of 2^(m_p - M) O_p, the same for l; this
    // part's own values come from its registers (they equal what it stored).
    // The other parts' values are read in batches of 32 ahead of their use, so
    // that their round trips overlap.
    const float* sml = slots + 4 * DB * 16 * 64 + w * 128 + lane;
    float M = m_run;
    for (int p2 = 0; p2 < np; ++p2)
      if (p2 != part) M = fmaxf(M, load_dev(sml + (size_t)p2 * PF));
    float L = 0.0f;
    for (int p2 = 0; p2 < np; ++p2) {
      const float mq = p2 == part ? m_run : load_dev(sml + (size_t)p2 * PF);
      const float lq = p2 == part ? l_run : load_dev(sml + (size_t)p2 * PF + 64);
      L = fmaf(lq, exp2f(mq - M), L);
    }
    l_run = L;
    const float w_own = exp2f(m_run - M);
#pragma unroll
    for (int db = 0; db < DB; db += 2) {
      float acc[32];
#pragma unroll
      for (int i = 0; i < 32; ++i) acc[i] = 0.0f;
      for (int p2 = 0; p2 < np; ++p2) {
        float x[32];
        float wq;
        if (p2 == part) {
#pragma unroll
          for (int i = 0; i < 32; ++i) x[i] = o[db + (i >> 4)][i & 15];
          wq = w_own;
        } else {
          const float* so = slots + (size_t)p2 * PF + (size_t)w * DB * 16 * 64 + (size_t)db * 16 * 64 + lane;
#pragma unroll
          for (int i = 0; i < 32; ++i) x[i] = load_dev(so + i * 64);
          wq = exp2f(load_dev(sml + (size_t)p2 * PF) - M);
        }
#pragma unroll
        for (int i = 0; i < 32; ++i) acc[i] = fmaf(x[i], wq, acc[i]);
      }
#pragma unroll
      for (int i = 0; i < 32; ++i) o[db + (i >> 4)][i & 15] = acc[i];
    }
  }

  // out = O / l, one RNE rounding: lane = query, rows = dims 32 db + 8 (r / 4) + 4 hl + r % 4
  if (query < a.T) {
    const float inv = 1.0f / l_run;
    uint16_t* orow = static_cast<uint16_t*>(a.out) + ((size_t)b * a.T + query) * a.n_q * HD + (size_t)h * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        uint2 v;
        v.x = pack_bf16x2(o[db][4 * g4 + 0] * inv, o[db][4 * g4 + 1] * inv);
        v.y = pack_bf16x2(o[db][4 * g4 + 2] * inv, o[db][4 * g4 + 3] * inv);
        *reinterpret_cast<uint2*>(orow + 32 * db + 8 * g4 + 4 * hl) = v;
      }
  }
}

__global__ void fill_ones_kernel(uint16_t* dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = 0x3f80;  // 1.0 in bf16
}

__global__ void fill_zero_u64_kernel(unsigned long long* dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = 0ull;
}

// ------------------------------------------------------------------ launchers

// Raise a kernel's dynamic-LDS limit once per process; `done` is the largest
// size set so far (racing threads may both set the idempotent attribute).
template <class Kern>
static hipError_t set_lds_once(Kern k, size_t bytes, std::atomic<size_t>& done) {
  if (bytes <= done.load(std::memory_order_acquire)) return hipSuccess;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)bytes);
  if (e != hipSuccess) return e;
  size_t cur = done.load(std::memory_order_relaxed);
  while (cur < bytes && !done.compare_exchange_weak(cur, bytes, std::memory_order_release)) {
  }
  return hipSuccess;
}

template <int EPI, bool NORM, bool PACKED, int MT>
static hipError_t gemm_t(const GemmArgs& a, hipStream_t st) {
  const size_t bytes = gemm_lds_bytes(a.K, MT);
  static std::atomic<size_t> done{0};
  auto k = gemm_kernel<EPI, NORM, PACKED, MT>;
  hipError_t e = set_lds_once(k, bytes, done);
  if (e != hipSuccess) return e;
  const int n_tiles = (a.M + MT - 1) / MT;
  const int n_units = EPI == kEpiResidual ? a.N / 512 : a.N / 256;
  const XcdMap m = xcd_map((long long)n_units * n_tiles);
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(kNtTile), bytes, st, a, m.per, n_tiles, n_units);
  return hipGetLastError();
}

// 128-token tiles take about 1.4-1.5x a 64-token tile's time for twice its
// work (measured: the projections of a Gemma-3-4B-shaped block); the launch
// takes them when its rounds of the chip (kWideMinTiles workgroups each) then
// cost no more, and their LDS fits.
constexpr int kGemmWideCost2 = 3;  // twice the relative time of a 128-token tile
template <int EPI, bool NORM, bool PACKED>
static hipError_t gemm_mt(const GemmArgs& a, hipStream_t st) {
  const long long units = EPI == kEpiResidual ? a.N / 512 : a.N / 256;
  const long long r64 = (units * ((a.M + kMtBf16 - 1) / kMtBf16) + kWideMinTiles - 1) / kWideMinTiles;
  const long long r128 = (units * ((a.M + 2LL * kMtBf16 - 1) / (2 * kMtBf16)) + kWideMinTiles - 1) / kWideMinTiles;
  const bool wide = kGemmWideCost2 * r128 <= 2 * r64 && gemm_lds_bytes(a.K, 2 * kMtBf16) <= kLdsPerGroup;
  return wide ? gemm_t<EPI, NORM, PACKED, 2 * kMtBf16>(a, st) : gemm_t<EPI, NORM, PACKED, kMtBf16>(a, st);
}

hipError_t launch_gemm(const GemmArgs& a, int epi, int packed, hipStream_t st) {
  if (epi == kEpiResidual) {
    if (a.norm) return packed ? gemm_mt<kEpiResidual, true, true>(a, st) : gemm_mt<kEpiResidual, true, false>(a, st);
    return packed ? gemm_mt<kEpiResidual, false, true>(a, st) : gemm_mt<kEpiResidual, false, false>(a, st);
  }
  if (a.norm) return packed ? gemm_mt<kEpiSwiglu, true, true>(a, st) : gemm_mt<kEpiSwiglu, true, false>(a, st);
  return packed ? gemm_mt<kEpiSwiglu, false, true>(a, st) : gemm_mt<kEpiSwiglu, false, false>(a, st);
}

template <int HD>
static hipError_t prefill_t(const PrefillArgs& a, hipStream_t st) {
  constexpr size_t bytes = prefill_lds(HD).end;
  static std::atomic<size_t> done{0};
  auto k = prefill_attn_kernel<HD>;
  hipError_t e = set_lds_once(k, bytes, done);
  if (e != hipSuccess) return e;
  const long long pieces = a.n_order > 0 ? a.n_order : (a.T + 127) / 128;
  const long long items = (long long)a.B * a.n_q * pieces;
  hipLaunchKernelGGL(k, dim3((unsigned)items), dim3(256), bytes, st, a);
  return hipGetLastError();
}

// The split aims at about kPrefillTargetCus workgroups' worth of equal work:
// P = max(8, ceil(total key blocks / target)) key blocks per part, so a launch
// whose blocks already fill the chip (long batches, many heads) splits nothing.
constexpr long long kPrefillTargetCus = 256;
PrefillSplit prefill_split(int B, int T, int n_q) {
  PrefillSplit sp{};
  sp.P = 1;
  sp.NP = 1;
  if (B <= 0 || T <= 0) return sp;
  const int nqb = (T + 127) / 128;
  auto nkb = [&](int qb) { return (int)(std::min(128LL * qb + 127, (long long)T - 1) / 64 + 1); };
  long long per_head = 0;
  for (int qb = 0; qb < nqb; ++qb) per_head += nkb(qb);
  const long long total = per_head * B * n_q;
  const long long nkb_max = nkb(nqb - 1);
  sp.P = (int)std::min<long long>(std::max(8LL, (total + kPrefillTargetCus - 1) / kPrefillTargetCus), nkb_max);
  sp.NP = (int)((nkb_max + sp.P - 1) / sp.P);
  // the pieces of one head, longest first (ties: the later block first)
  struct Piece {
    int len, qb, part;
  };
  Piece pc[kPrefillOrderMax];
  int n = 0;
  for (int qb = nqb - 1; qb >= 0; --qb) {
    const int nk = nkb(qb), np = (nk + sp.P - 1) / sp.P;
    for (int p = 0; p < np; ++p) {
      if (n == kPrefillOrderMax || sp.NP > 255) {
        // too many pieces to list: no split, blocks from the last
        sp.P = (int)nkb_max;
        sp.NP = 1;
        sp.n_order = 0;
        return sp;
      }
      pc[n++] = Piece{(p + 1) * nk / np - p * nk / np, qb, p};
    }
  }
  std::stable_sort(pc, pc + n, [](const Piece& x, const Piece& y) { return x.len > y.len; });
  sp.n_order = n;
  for (int i = 0; i < n; ++i) sp.order[i] = ((unsigned)pc[i].qb << 8) | (unsigned)pc[i].part;
  return sp;
}

size_t prefill_part_floats(int hd) { return (size_t)4 * ((hd / 32) * 16 * 64 + 128); }

size_t prefill_lds_bytes(int hd) { return prefill_lds(hd).end; }
size_t gemm_lds_bytes(int K, int mt) { return proj_lds<uint16_t>(256, mt).end + gamma_lds_bytes(K); }

hipError_t launch_prefill_attn(const PrefillArgs& a, int hd, hipStream_t st) {
  switch (hd) {
    case 128: return prefill_t<128>(a, st);
    case 256: return prefill_t<256>(a, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fill_ones_bf16(void* dst, int n, hipStream_t st) {
  hipLaunchKernelGGL(fill_ones_kernel, dim3((n + 255) / 256), dim3(256), 0, st, static_cast<uint16_t*>(dst), n);
  return hipGetLastError();
}

hipError_t launch_fill_zero_u64(void* dst, int n, hipStream_t st) {
  hipLaunchKernelGGL(fill_zero_u64_kernel, dim3((n + 255) / 256), dim3(256), 0, st,
                     static_cast<unsigned long long*>(dst), n);
  return hipGetLastError();
}

}  // namespace kvd
