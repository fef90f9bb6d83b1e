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
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvd_layout.h"

namespace kvd {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

template <int N> struct IC { static constexpr int value = N; };

// ------------------------------------------------------------------ scalars

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  __bf16 x = (__bf16)a;  // round to nearest even
  __bf16 y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
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

// Per-token 1/rms from the per-thread partial sums: thread (row, sub) holds the
// sum over its chunk column sub = tid & 7; the 8 partials of a row sit in 8
// consecutive lanes and are added by a fixed xor tree.
template <int CPT>
__device__ __forceinline__ void finish_rms(const float (&ss)[CPT], const bool (&valid)[CPT], int d, float eps,
                                           float* rinv) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int r = 0; r < CPT; ++r) {
    float v = ss[r];
    v += __shfl_xor(v, 1, 64);
    v += __shfl_xor(v, 2, 64);
    v += __shfl_xor(v, 4, 64);
    if ((tid & 7) == 0) rinv[(tid >> 3) + 32 * r] = valid[r] ? 1.0f / sqrtf(v / (float)d + eps) : 0.0f;
  }
}

// One half (head_dim rows) of a projection tile: the weight block it reads, whether
// its rows get RoPE, and its column offset in the LDS K/V tile (0 or head_dim).
struct Half {
  const void* w;  // first row of a [head_dim][d] block, or nullptr (rows absent -> zeros)
  int rope;
};

// ------------------------------------------------------------------ bf16 MFMA tile

template <int HD, int MT>
struct MfmaTile {
  static constexpr int NB_F = HD >= 128 ? HD / 64 : 1;  // 32-row blocks per wave
  static constexpr int NB_T = MT / 32;                  // 32-token blocks
  static constexpr int CPT = MT / 32;                   // staged chunks per thread per K-step
  static constexpr int HLD = h_ld<uint16_t>();
  static constexpr int KLD = kv_ld<uint16_t>(HD);

  // Rows covered by block bf of wave w: which half (K/first = 0, V/second = 1) and
  // the first row inside that half.  head_dim >= 128: every wave owns head_dim/4
  // rows of each half; head_dim == 64: waves 0-1 own the first half, 2-3 the second.
  static __device__ __forceinline__ void block_rows(int wave, int bf, int& half, int& row0) {
    if (HD == 64) {
      half = wave >> 1;
      row0 = 32 * (wave & 1);
    } else {
      constexpr int hb = NB_F / 2;
      half = bf / hb;
      row0 = (HD / 4) * wave + 32 * (bf % hb);
    }
  }

  // Computes the tile into `kv` (LDS, [MT][KLD] bf16): rows of half 0 at columns
  // 0..HD-1, half 1 at HD..2HD-1.  hrow[r]: residual row of staged token
  // (tid>>3)+32r, already offset by 8*(tid&7), or nullptr for a padding token.
  // pos (LDS [MT]) and rev (LDS [HD/2]) feed RoPE; rinv is LDS scratch [MT].
  static __device__ void run(const uint16_t* const (&hrow)[CPT], const uint16_t* gamma, int d, float eps,
                             const Half (&halves)[2], uint16_t* hst, float* rinv, const int* pos,
                             const double* rev, uint16_t* kv) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, sub = tid & 7;
    const int nsteps = d / kKT;

    const uint16_t* wrow[NB_F];
#pragma unroll
    for (int bf = 0; bf < NB_F; ++bf) {
      int half, row0;
      block_rows(wave, bf, half, row0);
      const uint16_t* w = static_cast<const uint16_t*>(halves[half].w);
      wrow[bf] = w ? w + (size_t)(row0 + (lane & 31)) * d + 8 * (lane >> 5) : nullptr;
    }
    bool valid[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) valid[r] = hrow[r] != nullptr;

    f32x16_t acc[NB_F][NB_T];
#pragma unroll
    for (int bf = 0; bf < NB_F; ++bf)
#pragma unroll
      for (int bt = 0; bt < NB_T; ++bt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[bf][bt][i] = 0.0f;

    bf16x8_t a[2][NB_F][4];
    uint4 hv[CPT];
    uint4 gv;
    float ss[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) ss[r] = 0.0f;

    auto load_h = [&](int s) {
#pragma unroll
      for (int r = 0; r < CPT; ++r)
        hv[r] = valid[r] ? *reinterpret_cast<const uint4*>(hrow[r] + (size_t)s * kKT) : make_uint4(0, 0, 0, 0);
      gv = *reinterpret_cast<const uint4*>(gamma + (size_t)s * kKT + 8 * sub);
    };
    auto store_h = [&](int buf) {
#pragma unroll
      for (int r = 0; r < CPT; ++r) {
        const uint4 o = stage_chunk_bf16(hv[r], gv, ss[r]);
        *reinterpret_cast<uint4*>(hst + ((size_t)buf * MT + (tid >> 3) + 32 * r) * HLD + 8 * sub) = o;
      }
    };
    auto load_a = [&](auto buf_c, int s) {
      constexpr int B = decltype(buf_c)::value;
#pragma unroll
      for (int bf = 0; bf < NB_F; ++bf)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (wrow[bf]) {
            a[B][bf][u] = *reinterpret_cast<const bf16x8_t*>(wrow[bf] + (size_t)s * kKT + 16 * u);
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) a[B][bf][u][i] = (__bf16)0.0f;
          }
        }
    };
    auto kstep = [&](auto cur_c, int s) {
      constexpr int C = decltype(cur_c)::value;
      const bool more = s + 1 < nsteps;
      if (more) {
        load_h(s + 1);
        load_a(IC<C ^ 1>{}, s + 1);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        bf16x8_t bv[NB_T];
#pragma unroll
        for (int bt = 0; bt < NB_T; ++bt)
          bv[bt] = *reinterpret_cast<const bf16x8_t*>(
              hst + ((size_t)C * MT + 32 * bt + (lane & 31)) * HLD + 16 * u + 8 * (lane >> 5));
#pragma unroll
        for (int bf = 0; bf < NB_F; ++bf)
#pragma unroll
          for (int bt = 0; bt < NB_T; ++bt)
            acc[bf][bt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[C][bf][u], bv[bt], acc[bf][bt], 0, 0, 0);
      }
      if (more) store_h(C ^ 1);
      __syncthreads();
    };

    load_h(0);
    load_a(IC<0>{}, 0);
    store_h(0);
    __syncthreads();
    for (int s = 0; s < nsteps; s += 2) {
      kstep(IC<0>{}, s);
      if (s + 1 < nsteps) kstep(IC<1>{}, s + 1);
    }

    finish_rms<CPT>(ss, valid, d, eps, rinv);
    __syncthreads();

    // epilogue: row scale, RoPE on rotated halves, one RNE rounding, LDS tile.
#pragma unroll
    for (int bt = 0; bt < NB_T; ++bt) {
      const int tok = 32 * bt + (lane & 31);
      const float ri = rinv[tok];
      const int p = pos[tok];
#pragma unroll
      for (int bf = 0; bf < NB_F; ++bf) {
        int half, row0;
        block_rows(wave, bf, half, row0);
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = acc[bf][bt][r] * ri;
        if (halves[half].rope) {
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
};

// ------------------------------------------------------------------ fp32 VALU tile

template <int HD, int MT>
struct F32Tile {
  static constexpr int TG = kThreads / HD;   // token groups
  static constexpr int TPT = MT / TG;        // tokens per thread
  static constexpr int CPT = MT / 32;
  static constexpr int HLD = h_ld<float>();
  static constexpr int KLD = kv_ld<float>(HD);

  static __device__ void run(const float* const (&hrow)[CPT], const float* gamma, int d, float eps,
                             const Half (&halves)[2], float* hst, float* rinv, const int* pos, const double* rev,
                             float* kv) {
    const int tid = threadIdx.x, sub = tid & 7;
    const int p = tid % HD;            // feature pair: rows 2p, 2p+1 of the 2*HD rows
    const int tg = tid / HD;
    const int half = (2 * p) / HD;
    const int r0 = (2 * p) % HD;
    const float* w = static_cast<const float*>(halves[half].w);
    const float* w0 = w ? w + (size_t)r0 * d : nullptr;
    const int nsteps = d / kKT;

    bool valid[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) valid[r] = hrow[r] != nullptr;
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
        if (valid[r]) {
          load8(hrow[r] + (size_t)s * kKT, x);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = 0.0f;
        }
        float* dst = hst + (size_t)((tid >> 3) + 32 * r) * HLD + 8 * sub;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          ss[r] = fmaf(x[e], x[e], ss[r]);
          dst[e] = x[e] * g[e];
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

    finish_rms<CPT>(ss, valid, d, eps, rinv);
    __syncthreads();

#pragma unroll
    for (int t = 0; t < TPT; ++t) {
      const int tok = tg * TPT + t;
      const float ri = rinv[tok];
      float v0 = acc0[t] * ri, v1 = acc1[t] * ri;
      if (halves[half].rope) rope_rotate(v0, v1, pos[tok], rev[r0 >> 1]);
      *reinterpret_cast<float2*>(kv + (size_t)tok * KLD + half * HD + r0) = make_float2(v0, v1);
    }
  }
};

// ------------------------------------------------------------------ attention

// q heads j*g .. j*g+g-1 of sequence b into LDS (fp32), pre-multiplied by
// log2(e)/sqrt(head_dim).
template <typename T, int HD>
__device__ __forceinline__ void load_q(const T* q, int b, int n_q, int j, int g, float* qs) {
  const T* src = q + ((size_t)b * n_q + (size_t)j * g) * HD;
  for (int i = threadIdx.x; i < g * HD; i += kThreads) qs[i] = to_f<T>(src[i]) * ScoreScale<HD>::v;
}

// Rows t0 .. t0+n-1 of a stored K/V block ([B][n_kv][t_cap][HD], head j of
// sequence b, rows counted from t_off) into the LDS tile [kTile][K | V].
template <typename T, int HD>
__device__ __forceinline__ void load_kv_tile(const T* K, const T* V, int b, int n_kv, int j, int t_cap, int row0,
                                             int n, T* kv) {
  constexpr int KLD = kv_ld<T>(HD);
  constexpr int CH = 16 / sizeof(T);  // elements per 16-byte chunk
  constexpr int CPR = HD / CH;        // chunks per K (or V) row
  const size_t base = ((size_t)b * n_kv + j) * t_cap + row0;
  for (int c = threadIdx.x; c < 2 * n * CPR; c += kThreads) {
    const int which = c / (n * CPR);  // 0: K, 1: V
    const int rem = c - which * n * CPR;
    const int t = rem / CPR, ch = rem - t * CPR;
    const T* src = (which ? V : K) + (base + t) * HD + ch * CH;
    *reinterpret_cast<uint4*>(kv + (size_t)t * KLD + which * HD + ch * CH) = *reinterpret_cast<const uint4*>(src);
  }
}

// Softmax partial state of keys 0..n-1 of an LDS K/V tile (rows stride KLD,
// K at columns 0..HD-1, V at HD..2HD-1) for g query heads:
//   m_h = max_t s_ht,  l_h = sum_t 2^(s_ht - m_h),  acc_h = sum_t 2^(s_ht - m_h) V_t,
// with s_ht = log2(e) q_h.K_t / sqrt(HD).  Results in LDS (L.ml, L.acc).
template <typename T, int HD>
__device__ void attend_tile(const T* kv, int n, int rows, int g, char* lds, const AttnLds& L) {
  constexpr int KLD = kv_ld<T>(HD);
  constexpr int C8 = HD / 8;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* qs = reinterpret_cast<const float*>(lds + L.q);
  float* S = reinterpret_cast<float*>(lds + L.s);
  float* red = reinterpret_cast<float*>(lds + L.red);
  float* ml = reinterpret_cast<float*>(lds + L.ml);
  float* acc = reinterpret_cast<float*>(lds + L.acc);

  for (int task = tid; task < g * rows; task += kThreads) {
    const int h = task / rows, t = task - h * rows;
    float s = -INFINITY;
    if (t < n) {
      const T* krow = kv + (size_t)t * KLD;
      const float* qh = qs + h * HD;
      float dot = 0.0f;
#pragma unroll 4
      for (int c = 0; c < C8; ++c) {
        float k8[8];
        load8(krow + 8 * c, k8);
        const float4 qa = *reinterpret_cast<const float4*>(qh + 8 * c);
        const float4 qb = *reinterpret_cast<const float4*>(qh + 8 * c + 4);
        dot = fmaf(qa.x, k8[0], dot);
        dot = fmaf(qa.y, k8[1], dot);
        dot = fmaf(qa.z, k8[2], dot);
        dot = fmaf(qa.w, k8[3], dot);
        dot = fmaf(qb.x, k8[4], dot);
        dot = fmaf(qb.y, k8[5], dot);
        dot = fmaf(qb.z, k8[6], dot);
        dot = fmaf(qb.w, k8[7], dot);
      }
      s = dot;
    }
    S[h * rows + t] = s;
  }
  __syncthreads();

  for (int h = wave; h < g; h += kThreads / 64) {
    float m = -INFINITY;
    for (int t = lane; t < n; t += 64) m = fmaxf(m, S[h * rows + t]);
    m = wave_max(m);
    float l = 0.0f;
    for (int t = lane; t < rows; t += 64) {
      const float p = t < n ? exp2f(S[h * rows + t] - m) : 0.0f;
      S[h * rows + t] = p;
      l += p;
    }
    l = wave_sum(l);
    if (lane == 0) {
      ml[2 * h] = m;
      ml[2 * h + 1] = l;
    }
  }
  __syncthreads();

  const int per = g * C8;
  const int TS = per >= kThreads ? 1 : kThreads / per;
  for (int task = tid; task < TS * per; task += kThreads) {
    const int c8 = task % C8;
    const int rest = task / C8;
    const int h = rest % g, ts = rest / g;
    float a8[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int t = ts; t < n; t += TS) {
      const float p = S[h * rows + t];
      float v8[8];
      load8(kv + (size_t)t * KLD + HD + 8 * c8, v8);
#pragma unroll
      for (int e = 0; e < 8; ++e) a8[e] = fmaf(p, v8[e], a8[e]);
    }
    float* dst = red + ((size_t)ts * g + h) * HD + 8 * c8;
#pragma unroll
    for (int e = 0; e < 8; ++e) dst[e] = a8[e];
  }
  __syncthreads();
  for (int idx = tid; idx < g * HD; idx += kThreads) {
    float s = 0.0f;
    for (int ts = 0; ts < TS; ++ts) s += red[(size_t)ts * g * HD + idx];
    acc[idx] = s;
  }
  __syncthreads();
}

// Split-K partial of (b, KV head j, split s) into the workspace:
// acc [B][n_q][S][HD] fp32 followed by ml [B][n_q][S][2] fp32.
template <int HD>
__device__ __forceinline__ void write_partial(const char* lds, const AttnLds& L, float* ws_acc, float* ws_ml, int b,
                                              int n_q, int j, int g, int S, int s) {
  const float* acc = reinterpret_cast<const float*>(lds + L.acc);
  const float* ml = reinterpret_cast<const float*>(lds + L.ml);
  for (int idx = threadIdx.x; idx < g * HD; idx += kThreads) {
    const int h = idx / HD, c = idx - h * HD;
    ws_acc[(((size_t)b * n_q + (size_t)j * g + h) * S + s) * HD + c] = acc[idx];
  }
  if (threadIdx.x < 2 * g) {
    const int h = threadIdx.x >> 1, k = threadIdx.x & 1;
    ws_ml[(((size_t)b * n_q + (size_t)j * g + h) * S + s) * 2 + k] = ml[threadIdx.x];
  }
}

}  // namespace kvd
