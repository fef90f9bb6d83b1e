// Kernels of the single-checkpoint scheme: one pre-norm transformer block over
// all positions (Sec. 3.1, Eqs. q_proj .. mlp_sublayer), run layer after layer
// to recompute h^(l) from the one stored residual per token (Eq. res_mem).
// The Q/K/V projections are the recompute tile engine's (proj_kernel); this file
// holds the output projections (W_o, and the MLP's gate/up and down) on the same
// MFMA tile engine with other epilogues, and causal prefill attention.
#include <hip/hip_runtime.h>

#include "kvd_device.hpp"
#include "kvd_launch.h"

namespace kvd {

// ------------------------------------------------------------------ projections with residual / SwiGLU epilogues

// grid: xcd_map(n_units * n_tiles) workgroups; item = unit * n_tiles + tile (the
// token tiles of one weight block run on one XCD).  A unit is 512 rows of W
// (kEpiResidual) or 256 rows each of W and W2 (kEpiSwiglu); a tile is 64 token rows.
template <int EPI, bool NORM, bool PACKED>
__global__ __launch_bounds__(kNtTile, 1) void gemm_kernel(GemmArgs a, int per_xcd, int n_tiles, int n_units) {
  extern __shared__ __align__(16) char lds[];
  constexpr int NT = kNtTile, HD = 256, MT = kMtBf16;
  constexpr ProjLds PL = proj_lds<uint16_t>(HD, MT);
  constexpr int KLD = kv_ld<uint16_t>(HD);
  using Tile = MfmaTile<HD, MT, PACKED>;
  static_assert(Tile::NB_F == 2 && Tile::WT == 1 && Tile::NB_T == 2, "wave fw owns rows 32 fw.. of both halves");
  const int tid = threadIdx.x;
  const long long item = (long long)(blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (item >= (long long)n_units * n_tiles) return;
  const int unit = (int)(item / n_tiles);
  const int tile = (int)(item - (long long)unit * n_tiles);
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
  Tile::run_with(hrow, valid, gam, gsrc, a.K, a.eps, halves, hst, rinv, setup,
                 [&](const f32x16_t (&acc)[2][2], const bool (&)[2]) {
#pragma unroll
                   for (int bt = 0; bt < 2; ++bt) {
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
                 });
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

// LDS of prefill_attn_kernel (bytes): the key tile [64][HD + 8] bf16, the value
// tile transposed [HD][64 + 8] bf16, scores [64][65] fp32, probabilities
// [64][64 + 8] bf16, and per query row the running max, sum and rescale factor.
struct PrefillLds {
  size_t ks, vt, ss, ps, m, l, al, end;
};
constexpr PrefillLds prefill_lds(int hd) {
  PrefillLds L{};
  L.ks = 0;
  L.vt = L.ks + (size_t)2 * 64 * (hd + 8);
  L.ss = L.vt + (size_t)2 * hd * (64 + 8);
  L.ps = L.ss + (size_t)4 * 64 * 65;
  L.m = L.ps + (size_t)2 * 64 * (64 + 8);
  L.l = L.m + 4 * 64;
  L.al = L.l + 4 * 64;
  L.end = L.al + 4 * 64;
  return L;
}

// grid: xcd_map(B * n_q * nqb) workgroups, nqb = ceil(T / 64), 256 threads (4
// waves).  Items are ordered (sequence, KV head, query block from the last,
// query head of the group), so an XCD's workgroups share one KV head's keys and
// values in its L2 and the longest rows start first.  A workgroup takes 64 query
// rows of one head through the key blocks 0 .. its own (flash order: scores,
// running max / sum, rescaled accumulators), loading key block kb + 1 into
// registers while block kb is computed.  Wave w computes the 32 x 32 score block
// (query half w / 2, key half w % 2) with its query rows in registers, and the
// output columns [w % 2 * hd / 2, + hd / 2) of query half w / 2.  Scores are in
// the log2 domain (log2(e) / sqrt(hd) folded into the scale).
template <int HD>
__global__ __launch_bounds__(256) void prefill_attn_kernel(PrefillArgs a, int per_xcd) {
  extern __shared__ __align__(16) char lds[];
  constexpr PrefillLds PL = prefill_lds(HD);
  constexpr int KS = HD / 16;   // 16-wide k-steps of a score block
  constexpr int DBW = HD / 64;  // 32-wide output column blocks per wave
  constexpr int KLDS = HD + 8, VLD = 64 + 8, SLD = 65, PLD = 64 + 8;
  constexpr int CPR = HD / 8;              // 16-byte chunks per key row
  constexpr int KCH = 64 * CPR / 256;      // key chunks per thread
  constexpr int VGR = 16 * CPR / 256;      // value groups (4 keys x 8 columns) per thread
  uint16_t* Ks = reinterpret_cast<uint16_t*>(lds + PL.ks);
  uint16_t* Vt = reinterpret_cast<uint16_t*>(lds + PL.vt);
  float* Ss = reinterpret_cast<float*>(lds + PL.ss);
  uint16_t* Ps = reinterpret_cast<uint16_t*>(lds + PL.ps);
  float* mrow = reinterpret_cast<float*>(lds + PL.m);
  float* lrow = reinterpret_cast<float*>(lds + PL.l);
  float* arow = reinterpret_cast<float*>(lds + PL.al);

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int nqb = (a.T + 63) / 64;
  const int g = a.n_q / a.n_kv;
  const long long item = (long long)(blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (item >= (long long)a.B * a.n_q * nqb) return;
  const int hh = (int)(item % g);
  const long long r1 = item / g;
  const int qb = nqb - 1 - (int)(r1 % nqb);  // the longest rows first
  const long long r2 = r1 / nqb;
  const int j = (int)(r2 % a.n_kv), b = (int)(r2 / a.n_kv);
  const int h = j * g + hh;
  const int qi = w >> 1, kj = w & 1;
  const float scale = ScoreScale<HD>::v;
  const uint16_t* kbase = static_cast<const uint16_t*>(a.k) + ((size_t)b * a.n_kv + j) * a.T * HD;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + ((size_t)b * a.n_kv + j) * a.T * HD;

  // this wave's query rows as MFMA A operands: row 64 qb + 32 qi + lane % 32
  bf16x8_t qf[KS];
  {
    const int t = min(64 * qb + 32 * qi + (lane & 31), a.T - 1);
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + (((size_t)b * a.T + t) * a.n_q + h) * HD + 8 * (lane >> 5);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8_t*>(qrow + 16 * ks);
  }
  if (tid < 64) {
    mrow[tid] = -INFINITY;
    lrow[tid] = 0.0f;
  }
  f32x16_t o[DBW];
#pragma unroll
  for (int db = 0; db < DBW; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.0f;

  // key / value block kb into registers (rows clamped to T - 1: masked below)
  u32x4_t kc[KCH], vc[VGR][4];
  auto load_kv = [&](int kb) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + 256 * i, row = c / CPR, ch = c - row * CPR;
      const int t = min(64 * kb + row, a.T - 1);
      kc[i] = *reinterpret_cast<const u32x4_t*>(kbase + (size_t)t * HD + 8 * ch);
    }
#pragma unroll
    for (int i = 0; i < VGR; ++i) {
      const int gidx = tid + 256 * i, k4 = gidx & 15, ch = gidx >> 4;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int t = min(64 * kb + 4 * k4 + kk, a.T - 1);
        vc[i][kk] = *reinterpret_cast<const u32x4_t*>(vbase + (size_t)t * HD + 8 * ch);
      }
    }
  };
  load_kv(0);

  for (int kb = 0; kb <= qb; ++kb) {
    // the registers into LDS: K as is, V transposed ([column][key])
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + 256 * i, row = c / CPR, ch = c - row * CPR;
      *reinterpret_cast<u32x4_t*>(Ks + row * KLDS + 8 * ch) = kc[i];
    }
#pragma unroll
    for (int i = 0; i < VGR; ++i) {
      const int gidx = tid + 256 * i, k4 = gidx & 15, ch = gidx >> 4;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int word = e >> 1, sh = (e & 1) * 16;
        uint2 pk;
        pk.x = ((vc[i][0][word] >> sh) & 0xffffu) | (((vc[i][1][word] >> sh) & 0xffffu) << 16);
        pk.y = ((vc[i][2][word] >> sh) & 0xffffu) | (((vc[i][3][word] >> sh) & 0xffffu) << 16);
        *reinterpret_cast<uint2*>(Vt + (8 * ch + e) * VLD + 4 * k4) = pk;
      }
    }
    __syncthreads();
    if (kb < qb) load_kv(kb + 1);  // in flight while this block is computed

    // scores of block (qi, kj), masked, into LDS (two accumulators halve the chain)
    {
      f32x16_t s0, s1;
#pragma unroll
      for (int i = 0; i < 16; ++i) s0[i] = s1[i] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ks += 2) {
        const uint16_t* kr = Ks + (32 * kj + (lane & 31)) * KLDS + 8 * (lane >> 5);
        const bf16x8_t k0 = *reinterpret_cast<const bf16x8_t*>(kr + 16 * ks);
        const bf16x8_t k1 = *reinterpret_cast<const bf16x8_t*>(kr + 16 * ks + 16);
        s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[ks], k0, s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[ks + 1], k1, s1, 0, 0, 0);
      }
      const int key = 64 * kb + 32 * kj + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = 32 * qi + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int query = 64 * qb + rl;
        float v = (s0[r] + s1[r]) * scale;
        if (query >= a.T) v = 0.0f;  // rows past the end: finite, never stored
        else if (key > query) v = -INFINITY;
        Ss[rl * SLD + 32 * kj + (lane & 31)] = v;
      }
    }
    __syncthreads();

    // running softmax: 4 threads per query row, 16 keys each
    {
      const int row = tid >> 2, part = tid & 3;
      float x[16];
      float mx = -INFINITY;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        x[e] = Ss[row * SLD + 16 * part + e];
        mx = fmaxf(mx, x[e]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
      const float m_old = mrow[row];
      const float m_new = fmaxf(m_old, mx);
      float sum = 0.0f;
      uint32_t pw[8];
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const float p0 = exp2f(x[e] - m_new), p1 = exp2f(x[e + 1] - m_new);
        pw[e >> 1] = pack_bf16x2(p0, p1);
        sum += bf_lo(pw[e >> 1]) + bf_hi(pw[e >> 1]);  // the rounded weights the MFMA uses
      }
      *reinterpret_cast<uint4*>(Ps + row * PLD + 16 * part) = make_uint4(pw[0], pw[1], pw[2], pw[3]);
      *reinterpret_cast<uint4*>(Ps + row * PLD + 16 * part + 8) = make_uint4(pw[4], pw[5], pw[6], pw[7]);
      sum += __shfl_xor(sum, 1, 64);
      sum += __shfl_xor(sum, 2, 64);
      if (part == 0) {
        const float al = exp2f(m_old - m_new);
        arow[row] = al;
        lrow[row] = lrow[row] * al + sum;
        mrow[row] = m_new;
      }
    }
    __syncthreads();

    // o = o * alpha + P V over this key block
#pragma unroll
    for (int db = 0; db < DBW; ++db) {
      const int col0 = 32 * (DBW * kj + db);
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= arow[32 * qi + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8_t pf = *reinterpret_cast<const bf16x8_t*>(Ps + (32 * qi + (lane & 31)) * PLD + 16 * ks + 8 * (lane >> 5));
        const bf16x8_t vf = *reinterpret_cast<const bf16x8_t*>(Vt + (col0 + (lane & 31)) * VLD + 16 * ks + 8 * (lane >> 5));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf, vf, o[db], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // out = o / l, one RNE rounding
  uint16_t* out = static_cast<uint16_t*>(a.out);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int rl = 32 * qi + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    const int t = 64 * qb + rl;
    if (t >= a.T) continue;
    const float inv = 1.0f / lrow[rl];
#pragma unroll
    for (int db = 0; db < DBW; ++db) {
      const int col = 32 * (DBW * kj + db) + (lane & 31);
      out[((size_t)b * a.T + t) * a.n_q * HD + (size_t)h * HD + col] =
          (uint16_t)(pack_bf16x2(o[db][r] * inv, 0.0f) & 0xffffu);
    }
  }
}

__global__ void fill_ones_kernel(uint16_t* dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = 0x3f80;  // 1.0 in bf16
}

// ------------------------------------------------------------------ launchers

template <class Kern>
static hipError_t set_lds_once(Kern k, size_t bytes, size_t& done) {
  if (bytes <= done) return hipSuccess;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)bytes);
  if (e == hipSuccess) done = bytes;
  return e;
}

template <int EPI, bool NORM, bool PACKED>
static hipError_t gemm_t(const GemmArgs& a, hipStream_t st) {
  const size_t bytes = proj_lds<uint16_t>(256, kMtBf16).end + gamma_lds_bytes(a.K);
  static size_t done = 0;
  auto k = gemm_kernel<EPI, NORM, PACKED>;
  hipError_t e = set_lds_once(k, bytes, done);
  if (e != hipSuccess) return e;
  const int n_tiles = (a.M + kMtBf16 - 1) / kMtBf16;
  const int n_units = EPI == kEpiResidual ? a.N / 512 : a.N / 256;
  const XcdMap m = xcd_map((long long)n_units * n_tiles);
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(kNtTile), bytes, st, a, m.per, n_tiles, n_units);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& a, int epi, int packed, hipStream_t st) {
  if (epi == kEpiResidual) {
    if (a.norm) return packed ? gemm_t<kEpiResidual, true, true>(a, st) : gemm_t<kEpiResidual, true, false>(a, st);
    return packed ? gemm_t<kEpiResidual, false, true>(a, st) : gemm_t<kEpiResidual, false, false>(a, st);
  }
  if (a.norm) return packed ? gemm_t<kEpiSwiglu, true, true>(a, st) : gemm_t<kEpiSwiglu, true, false>(a, st);
  return packed ? gemm_t<kEpiSwiglu, false, true>(a, st) : gemm_t<kEpiSwiglu, false, false>(a, st);
}

template <int HD>
static hipError_t prefill_t(const PrefillArgs& a, hipStream_t st) {
  constexpr size_t bytes = prefill_lds(HD).end;
  static size_t done = 0;
  auto k = prefill_attn_kernel<HD>;
  hipError_t e = set_lds_once(k, bytes, done);
  if (e != hipSuccess) return e;
  const XcdMap m = xcd_map((long long)a.B * a.n_q * ((a.T + 63) / 64));
  hipLaunchKernelGGL(k, dim3(m.grid), dim3(256), bytes, st, a, m.per);
  return hipGetLastError();
}

size_t prefill_lds_bytes(int hd) { return prefill_lds(hd).end; }
size_t gemm_lds_bytes(int K) { return proj_lds<uint16_t>(256, kMtBf16).end + gamma_lds_bytes(K); }

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

}  // namespace kvd
