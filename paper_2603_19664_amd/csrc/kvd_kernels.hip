// Kernels and launchers of libkvd (gfx950).
//
//   proj_kernel     RMSNorm + projection + RoPE of token tiles (RECOMPUTE_KV /
//                   prefill, and the current token's q, K_t, V_t of a decode step).
//   fused_kernel    per (b, KV head, 64-key chunk): recompute K/V of the chunk
//                   into LDS and emit its split-K softmax partial without writing
//                   K/V to HBM; extra chunks attend a stored tail (CONCAT).
//   decode_kernel   per (b, KV head, 64-key chunk) of stored K/V: split-K partial.
//   combine_kernel  merges the partials of each (b, query head) in split order.
#include <hip/hip_runtime.h>

#include "kvd_device.hpp"
#include "kvd_launch.h"

namespace kvd {

// ------------------------------------------------------------------ projection

template <typename T, int HD, int MT>
__global__ __launch_bounds__(kThreads, 1) void proj_kernel(ProjArgs a) {
  extern __shared__ __align__(16) char lds[];
  constexpr ProjLds PL = proj_lds<T>(HD, MT);
  constexpr int CPT = MT / 32;
  constexpr int KLD = kv_ld<T>(HD);
  const int tid = threadIdx.x;
  double* rev = reinterpret_cast<double*>(lds + PL.rev);
  float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
  int* pos = reinterpret_cast<int*>(lds + PL.pos);
  T* hst = reinterpret_cast<T*>(lds + PL.hst);
  T* kv = reinterpret_cast<T*>(lds + PL.kv);

  const long long ntok = (long long)a.B * a.T;
  const long long n0 = (long long)blockIdx.x * MT;
  const int unit = blockIdx.y;
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

  if (tid < HD / 2) rev[tid] = a.rev[tid];
  if (tid < MT) {
    const long long n = n0 + tid;
    int p = 0;
    if (n < ntok) {
      const int b = (int)(n / a.T), t = (int)(n - (long long)b * a.T);
      p = a.pos0[b] + t;
    }
    pos[tid] = p;
  }
  const T* hrow[CPT];
#pragma unroll
  for (int r = 0; r < CPT; ++r) {
    const long long n = n0 + (tid >> 3) + 32 * r;
    if (n < ntok) {
      const int b = (int)(n / a.T), t = (int)(n - (long long)b * a.T);
      hrow[r] = static_cast<const T*>(a.h) + ((size_t)b * a.h_ld + t) * a.d + 8 * (tid & 7);
    } else {
      hrow[r] = nullptr;
    }
  }
  __syncthreads();

  if constexpr (sizeof(T) == 2) {
    MfmaTile<HD, MT>::run(hrow, static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves, hst, rinv, pos, rev, kv);
  } else {
    F32Tile<HD, MT>::run(hrow, static_cast<const float*>(a.gamma), a.d, a.eps, halves, hst, rinv, pos, rev, kv);
  }
  __syncthreads();

  // store: 16-byte chunks of each valid token row of each present half.
  constexpr int CH = 16 / sizeof(T);
  constexpr int CPR = HD / CH;
  for (int c = tid; c < 2 * MT * CPR; c += kThreads) {
    const int half = c / (MT * CPR);
    const int rem = c - half * MT * CPR;
    const int row = rem / CPR, ch = rem - row * CPR;
    const long long n = n0 + row;
    if (n >= ntok || halves[half].w == nullptr) continue;
    const int b = (int)(n / a.T), t = (int)(n - (long long)b * a.T);
    T* dst;
    if (kv_mode) {
      T* base = static_cast<T*>(half ? a.v_out : a.k_out);
      dst = base + (((size_t)b * a.n_kv + heads[half]) * a.kv_t_cap + a.kv_t_off + t) * HD;
    } else {
      dst = static_cast<T*>(a.q_out) + ((size_t)b * a.n_q + heads[half]) * HD;
    }
    *reinterpret_cast<uint4*>(dst + ch * CH) =
        *reinterpret_cast<const uint4*>(kv + (size_t)row * KLD + half * HD + ch * CH);
  }
}

// ------------------------------------------------------------------ fused recompute + attention

template <typename T, int HD, int MT>
__global__ __launch_bounds__(kThreads, 1) void fused_kernel(FusedArgs a) {
  extern __shared__ __align__(16) char lds[];
  constexpr ProjLds PL = proj_lds<T>(HD, MT);
  constexpr int CPT = MT / 32;
  constexpr int KLD = kv_ld<T>(HD);
  const int tid = threadIdx.x;
  const int s = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int g = a.n_q / a.n_kv;
  const AttnLds AL = attn_lds(PL.end, g, HD, MT);
  T* kv = reinterpret_cast<T*>(lds + PL.kv);

  load_q<T, HD>(static_cast<const T*>(a.q), b, a.n_q, j, g, reinterpret_cast<float*>(lds + AL.q));

  int n;
  if (s < a.n_rec) {
    const int t0 = s * MT;
    n = min(MT, a.T_rec - t0);
    double* rev = reinterpret_cast<double*>(lds + PL.rev);
    float* rinv = reinterpret_cast<float*>(lds + PL.rinv);
    int* pos = reinterpret_cast<int*>(lds + PL.pos);
    T* hst = reinterpret_cast<T*>(lds + PL.hst);
    if (tid < HD / 2) rev[tid] = a.rev[tid];
    if (tid < MT) pos[tid] = a.pos0[b] + t0 + tid;
    const T* hrow[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
      const int t = (tid >> 3) + 32 * r;
      hrow[r] = t < n ? static_cast<const T*>(a.h) + ((size_t)b * a.h_ld + t0 + t) * a.d + 8 * (tid & 7) : nullptr;
    }
    const size_t hd_d = (size_t)HD * a.d;
    const Half halves[2] = {Half{static_cast<const T*>(a.w_k) + j * hd_d, 1},
                            Half{static_cast<const T*>(a.w_v) + j * hd_d, 0}};
    __syncthreads();
    if constexpr (sizeof(T) == 2) {
      MfmaTile<HD, MT>::run(hrow, static_cast<const uint16_t*>(a.gamma), a.d, a.eps, halves, hst, rinv, pos, rev, kv);
    } else {
      F32Tile<HD, MT>::run(hrow, static_cast<const float*>(a.gamma), a.d, a.eps, halves, hst, rinv, pos, rev, kv);
    }
    __syncthreads();
    if (a.dbg_k != nullptr) {
      constexpr int CH = 16 / sizeof(T);
      constexpr int CPR = HD / CH;
      for (int c = tid; c < 2 * n * CPR; c += kThreads) {
        const int half = c / (n * CPR);
        const int rem = c - half * n * CPR;
        const int row = rem / CPR, ch = rem - row * CPR;
        T* base = static_cast<T*>(half ? a.dbg_v : a.dbg_k);
        T* dst = base + (((size_t)b * a.n_kv + j) * a.dbg_t_cap + a.dbg_t_off + t0 + row) * HD;
        *reinterpret_cast<uint4*>(dst + ch * CH) =
            *reinterpret_cast<const uint4*>(kv + (size_t)row * KLD + half * HD + ch * CH);
      }
    }
  } else {
    const int t0 = (s - a.n_rec) * MT;
    n = min(MT, a.T_tail - t0);
    load_kv_tile<T, HD>(static_cast<const T*>(a.tk), static_cast<const T*>(a.tv), b, a.n_kv, j, a.tail_t_cap,
                        a.tail_t_off + t0, n, kv);
    __syncthreads();
  }

  attend_tile<T, HD>(kv, n, MT, g, lds, AL);
  write_partial<HD>(lds, AL, a.ws_acc, a.ws_ml, b, a.n_q, j, g, a.S, s);
}

// ------------------------------------------------------------------ stored-K/V attention

template <typename T, int HD>
__global__ __launch_bounds__(kThreads) void decode_kernel(AttnArgs a) {
  extern __shared__ __align__(16) char lds[];
  const int s = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int g = a.n_q / a.n_kv;
  const AttnLds AL = attn_lds(align_up(sizeof(T) * kTile * kv_ld<T>(HD), 16), g, HD, kTile);
  T* kv = reinterpret_cast<T*>(lds);
  const int t0 = s * kTile;
  const int n = min(kTile, a.T - t0);
  load_q<T, HD>(static_cast<const T*>(a.q), b, a.n_q, j, g, reinterpret_cast<float*>(lds + AL.q));
  load_kv_tile<T, HD>(static_cast<const T*>(a.k), static_cast<const T*>(a.v), b, a.n_kv, j, a.t_cap, a.t_off + t0,
                      n, kv);
  __syncthreads();
  attend_tile<T, HD>(kv, n, kTile, g, lds, AL);
  write_partial<HD>(lds, AL, a.ws_acc, a.ws_ml, b, a.n_q, j, g, a.S, s);
}

// out[b][h] = sum_s 2^(m_s - M) acc_s / sum_s 2^(m_s - M) l_s, M = max_s m_s, in split order.
template <typename T, int HD>
__global__ __launch_bounds__(HD) void combine_kernel(const float* ws_acc, const float* ws_ml, T* out, int n_q, int S) {
  const int h = blockIdx.x, b = blockIdx.y, c = threadIdx.x;
  const size_t row = (size_t)b * n_q + h;
  const float* ml = ws_ml + row * S * 2;
  const float* acc = ws_acc + row * S * HD;
  float M = -INFINITY;
  for (int s = 0; s < S; ++s) M = fmaxf(M, ml[2 * s]);
  float L = 0.0f, o = 0.0f;
  for (int s = 0; s < S; ++s) {
    const float w = exp2f(ml[2 * s] - M);
    L = fmaf(ml[2 * s + 1], w, L);
    o = fmaf(acc[(size_t)s * HD + c], w, o);
  }
  out[row * HD + c] = from_f<T>(o / L);
}

// ------------------------------------------------------------------ launchers

template <typename K>
static hipError_t set_lds(K kernel, size_t bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

template <typename T, int HD>
static hipError_t proj_t(const ProjArgs& a, dim3 grid, hipStream_t st) {
  constexpr int MT = sizeof(T) == 2 ? kMtBf16 : kMtF32;
  constexpr size_t bytes = proj_lds<T>(HD, MT).end;
  auto k = proj_kernel<T, HD, MT>;
  hipError_t e = set_lds(k, bytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, grid, dim3(kThreads), bytes, st, a);
  return hipGetLastError();
}

template <typename T, int HD>
static hipError_t fused_t(const FusedArgs& a, dim3 grid, hipStream_t st) {
  constexpr int MT = sizeof(T) == 2 ? kMtBf16 : kMtF32;
  const size_t bytes = fused_lds_bytes<T>(a.n_q / a.n_kv, HD, MT);
  auto k = fused_kernel<T, HD, MT>;
  hipError_t e = set_lds(k, bytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, grid, dim3(kThreads), bytes, st, a);
  return hipGetLastError();
}

template <typename T, int HD>
static hipError_t attn_t(const AttnArgs& a, hipStream_t st) {
  const size_t bytes = decode_lds_bytes<T>(a.n_q / a.n_kv, HD);
  auto k = decode_kernel<T, HD>;
  hipError_t e = set_lds(k, bytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, dim3(a.S, a.n_kv, a.B), dim3(kThreads), bytes, st, a);
  e = hipGetLastError();
  if (e != hipSuccess || a.out == nullptr) return e;
  hipLaunchKernelGGL((combine_kernel<T, HD>), dim3(a.n_q, a.B), dim3(HD), 0, st, a.ws_acc, a.ws_ml,
                     static_cast<T*>(a.out), a.n_q, a.S);
  return hipGetLastError();
}

template <typename T, int HD>
static hipError_t combine_t(const float* ws_acc, const float* ws_ml, void* out, int n_q, int B, int S,
                            hipStream_t st) {
  hipLaunchKernelGGL((combine_kernel<T, HD>), dim3(n_q, B), dim3(HD), 0, st, ws_acc, ws_ml, static_cast<T*>(out),
                     n_q, S);
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

hipError_t launch_proj(const ProjArgs& a, int dtype_bf16, int hd, int n_units, hipStream_t st) {
  const int MT = dtype_bf16 ? kMtBf16 : kMtF32;
  const long long ntok = (long long)a.B * a.T;
  dim3 grid((unsigned)((ntok + MT - 1) / MT), (unsigned)n_units);
#define PB(H) proj_t<uint16_t, H>(a, grid, st)
#define PF(H) proj_t<float, H>(a, grid, st)
  KVD_DISPATCH(dtype_bf16, hd, PB, PF)
#undef PB
#undef PF
}

hipError_t launch_fused(const FusedArgs& a, int dtype_bf16, int hd, hipStream_t st) {
  dim3 grid((unsigned)a.S, (unsigned)a.n_kv, (unsigned)a.B);
  hipError_t e;
#define FB(H) fused_t<uint16_t, H>(a, grid, st)
#define FF(H) fused_t<float, H>(a, grid, st)
  e = [&]() -> hipError_t { KVD_DISPATCH(dtype_bf16, hd, FB, FF) }();
#undef FB
#undef FF
  if (e != hipSuccess || a.out == nullptr) return e;
  return launch_combine(a.ws_acc, a.ws_ml, a.out, a.n_q, a.B, a.S, dtype_bf16, hd, st);
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
#define AB(H) attn_t<uint16_t, H>(a, st)
#define AF(H) attn_t<float, H>(a, st)
  KVD_DISPATCH(dtype_bf16, hd, AB, AF)
#undef AB
#undef AF
}

}  // namespace kvd
