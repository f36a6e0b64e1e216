// Decode-step kernels: the projections of one token as matrix-vector products (each
// weight row is read once, so these are HBM-bound) with the epilogues of the prefill
// GEMMs, and the greedy pick over the vocabulary logits.
//
// One wave owns one item: a pair of weight rows whose results an epilogue needs together
// (the two rotary halves of a q / k dimension, the gate and up rows of one SwiGLU unit, or
// two neighbouring rows). Lanes stride the reduction axis by 8 elements, several 16-byte
// loads in flight per lane; the wave sum uses a fixed butterfly, so results are
// reproducible bit for bit.
#include "kernels.h"

namespace akvs {

namespace {

__device__ __forceinline__ float silu_dec(float g) { return g / (1.0f + __expf(-g)); }

// v rounded to the storage type T and widened back to fp32.
template <typename T>
__device__ __forceinline__ float load1_round(float v);
template <>
__device__ __forceinline__ float load1_round<float>(float v) { return v; }
template <>
__device__ __forceinline__ float load1_round<bf16_t>(float v) { return bf2f(f2bf(v)); }

// s0 = W[r0] . x, s1 = W[r1] . x over K (a multiple of 8), summed over the wave.
template <typename TW, typename TX>
__device__ __forceinline__ void dot2(const TW *__restrict__ w0, const TW *__restrict__ w1,
                                     const TX *__restrict__ x, int K, int lane, float &s0,
                                     float &s1) {
  constexpr int U = 4, STRIDE = 64 * 8;
  float a0 = 0.f, a1 = 0.f;
  int k = lane * 8;
  for (; k + (U - 1) * STRIDE < K; k += U * STRIDE) {
    float xv[U][8], wa[U][8], wb[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      load8(x + k + u * STRIDE, xv[u]);
      load8(w0 + k + u * STRIDE, wa[u]);
      load8(w1 + k + u * STRIDE, wb[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        a0 = fmaf(wa[u][i], xv[u][i], a0);
        a1 = fmaf(wb[u][i], xv[u][i], a1);
      }
  }
  for (; k < K; k += STRIDE) {
    float xv[8], wa[8], wb[8];
    load8(x + k, xv);
    load8(w0 + k, wa);
    load8(w1 + k, wb);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a0 = fmaf(wa[i], xv[i], a0);
      a1 = fmaf(wb[i], xv[i], a1);
    }
  }
  s0 = wave_sum(a0);
  s1 = wave_sum(a1);
}

template <typename TO>
__device__ __forceinline__ void put(void *base, size_t i, float v) {
  store1(reinterpret_cast<TO *>(base) + i, v);
}

__device__ __forceinline__ void put_dt(void *base, int dtype, size_t i, float v) {
  if (dtype == AKVS_BF16)
    put<bf16_t>(base, i, v);
  else
    put<float>(base, i, v);
}

// (value, index) order of the greedy pick: larger value first, equal values: lower index.
// Index -1 marks "none"; NaN values never win.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  if (i < 0 || v != v) return false;
  return bi < 0 || v > bv || (v == bv && i < bi);
}

// RMSNorm of the fp32 row h [K] into LDS: the arithmetic and summation order of k_rmsnorm
// (per-thread strided sums, fixed wave butterfly, waves added pairwise), so the normalised
// row equals what that kernel writes, rounded to TW.
template <typename TW>
__device__ __forceinline__ void norm_row_lds(const float *__restrict__ h, const TW *gain, int K,
                                             float eps, float *s_x) {
  __shared__ float red[4];
  float ss = 0.f;
  for (int e = threadIdx.x * 8; e < K; e += 256 * 8) {
    float v[8];
    load8(h + e, v);
#pragma unroll
    for (int k = 0; k < 8; ++k) ss = fmaf(v[k], v[k], ss);
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)K + eps);
  for (int e = threadIdx.x * 8; e < K; e += 256 * 8) {
    float v[8], g[8];
    load8(h + e, v);
    load8(gain + e, g);
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = load1_round<TW>(v[k] * inv * g[k]);
    store8(s_x + e, v);
  }
  __syncthreads();
}

template <typename TW, typename TX, bool NORM>
__global__ __launch_bounds__(256) void k_gemv(const TX *__restrict__ x,
                                              const TW *__restrict__ W, int N, int K,
                                              GemvEpi e) {
  __shared__ float s_val[4];
  __shared__ int s_idx[4];
  extern __shared__ float s_x[];  // NORM: the normalised row [K]
  if (NORM) {
    norm_row_lds(reinterpret_cast<const float *>(x), reinterpret_cast<const TW *>(e.norm), K,
                 e.eps, s_x);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long long item = (long long)blockIdx.x * 4 + wave;
  const long long n_items = (N + 1) / 2;
  const bool live = item < n_items;
  int r0 = 0, r1 = 0;
  if (live) {
    if (e.mode == GV_QKV) {
      const int half = e.hd >> 1;
      const int nq = e.hq_w >> 1, nk = e.kv_w >> 1;
      const int i = (int)item;
      if (i < nq) {
        r0 = (i / half) * e.hd + i % half;
        r1 = r0 + half;
      } else if (i < nq + nk) {
        const int j = i - nq;
        r0 = e.hq_w + (j / half) * e.hd + j % half;
        r1 = r0 + half;
      } else {
        r0 = e.hq_w + e.kv_w + 2 * (i - nq - nk);
        r1 = r0 + 1;
      }
    } else if (e.mode == GV_SWIGLU) {
      r0 = (int)item;       // gate row
      r1 = N / 2 + r0;      // up row
    } else {
      r0 = (int)(2 * item);
      r1 = min(r0 + 1, N - 1);
    }
  }
  float s0 = 0.f, s1 = 0.f;
  if (live) {
    if (NORM)
      dot2(W + (size_t)r0 * K, W + (size_t)r1 * K, static_cast<const float *>(s_x), K, lane, s0,
           s1);
    else
      dot2(W + (size_t)r0 * K, W + (size_t)r1 * K, x, K, lane, s0, s1);
  }
  if (e.mode == GV_LOGITS) {
    // both logits out, then the block's best (value, index) as a partial of the pick
    float bv = -INFINITY;
    int bi = -1;
    if (live) {
      if (lane == 0) {
        e.out_f32[r0] = s0;
        if (2 * item + 1 < N) e.out_f32[r1] = s1;
      }
      if (better(s0, r0, bv, bi)) { bv = s0; bi = r0; }
      if (2 * item + 1 < N && better(s1, r1, bv, bi)) { bv = s1; bi = r1; }
    }
    if (lane == 0) {
      s_val[wave] = bv;
      s_idx[wave] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      for (int w = 1; w < 4; ++w)
        if (better(s_val[w], s_idx[w], bv, bi)) { bv = s_val[w]; bi = s_idx[w]; }
      e.part_val[blockIdx.x] = bv;
      e.part_idx[blockIdx.x] = bi;
    }
    return;
  }
  if (!live || lane != 0) return;
  if (e.mode == GV_RESID) {
    e.out_f32[r0] += s0;
    if (2 * item + 1 < N) e.out_f32[r1] += s1;
  } else if (e.mode == GV_SWIGLU) {
    put_dt(e.out, e.out_dtype, r0, silu_dec(s0) * s1);
  } else {  // GV_QKV
    if (r0 < e.hq_w + e.kv_w) {
      const int half = e.hd >> 1;
      const float2 cs = e.rope[(r0 % e.hd) % half];
      const float lo = s0 * cs.x - s1 * cs.y;
      const float hi = s1 * cs.x + s0 * cs.y;
      if (r0 < e.hq_w) {
        put_dt(e.q_out, e.out_dtype, r0, lo);
        put_dt(e.q_out, e.out_dtype, r1, hi);
      } else {
        put_dt(e.k_out, e.out_dtype, r0 - e.hq_w, lo);
        put_dt(e.k_out, e.out_dtype, r1 - e.hq_w, hi);
      }
    } else {
      put_dt(e.v_out, e.out_dtype, r0 - e.hq_w - e.kv_w, s0);
      put_dt(e.v_out, e.out_dtype, r1 - e.hq_w - e.kv_w, s1);
    }
  }
}

// One block: the best (value, index) of n partials, in the order of `better`.
__global__ __launch_bounds__(256) void k_pick(const float *__restrict__ pv,
                                              const int32_t *__restrict__ pi, int n,
                                              int32_t *out) {
  __shared__ float s_val[256];
  __shared__ int s_idx[256];
  float bv = -INFINITY;
  int bi = -1;
  int i0 = threadIdx.x;
  for (; i0 + 7 * 256 < n; i0 += 8 * 256) {  // eight partials in flight per round trip
    float v[8];
    int ix[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      v[u] = pv[i0 + u * 256];
      ix[u] = pi[i0 + u * 256];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (better(v[u], ix[u], bv, bi)) { bv = v[u]; bi = ix[u]; }
  }
  for (; i0 < n; i0 += 256)
    if (better(pv[i0], pi[i0], bv, bi)) { bv = pv[i0]; bi = pi[i0]; }
  s_val[threadIdx.x] = bv;
  s_idx[threadIdx.x] = bi;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      const float v = s_val[threadIdx.x + o];
      const int i = s_idx[threadIdx.x + o];
      if (better(v, i, s_val[threadIdx.x], s_idx[threadIdx.x])) {
        s_val[threadIdx.x] = v;
        s_idx[threadIdx.x] = i;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = s_idx[0];
}

}  // namespace

int gemv_blocks(int N) { return (int)(((N + 1) / 2 + 3) / 4); }

hipError_t launch_gemv(const void *x, int x_dtype, const void *W, int w_dtype, int N, int K,
                       const GemvEpi &e, hipStream_t s) {
  if (N == 0) return hipSuccess;
  dim3 g((unsigned)gemv_blocks(N)), b(256);
  if (e.norm) {  // x: the fp32 residual row, normalised in each block
    if (x_dtype != AKVS_F32 || K > GEMV_NORM_MAX || K % 8) return hipErrorInvalidValue;
    const size_t lds = (size_t)K * sizeof(float);
    const float *h = reinterpret_cast<const float *>(x);
    if (w_dtype == AKVS_BF16)
      hipLaunchKernelGGL((k_gemv<bf16_t, float, true>), g, b, lds, s, h,
                         reinterpret_cast<const bf16_t *>(W), N, K, e);
    else
      hipLaunchKernelGGL((k_gemv<float, float, true>), g, b, lds, s, h,
                         reinterpret_cast<const float *>(W), N, K, e);
    return hipGetLastError();
  }
  if (w_dtype == AKVS_BF16) {
    const bf16_t *w = reinterpret_cast<const bf16_t *>(W);
    if (x_dtype == AKVS_BF16)
      hipLaunchKernelGGL((k_gemv<bf16_t, bf16_t, false>), g, b, 0, s,
                         reinterpret_cast<const bf16_t *>(x), w, N, K, e);
    else
      hipLaunchKernelGGL((k_gemv<bf16_t, float, false>), g, b, 0, s,
                         reinterpret_cast<const float *>(x), w, N, K, e);
  } else {
    const float *w = reinterpret_cast<const float *>(W);
    if (x_dtype == AKVS_BF16)
      hipLaunchKernelGGL((k_gemv<float, bf16_t, false>), g, b, 0, s,
                         reinterpret_cast<const bf16_t *>(x), w, N, K, e);
    else
      hipLaunchKernelGGL((k_gemv<float, float, false>), g, b, 0, s,
                         reinterpret_cast<const float *>(x), w, N, K, e);
  }
  return hipGetLastError();
}

hipError_t launch_pick(const float *part_val, const int32_t *part_idx, int n, int32_t *out,
                       hipStream_t s) {
  hipLaunchKernelGGL(k_pick, dim3(1), dim3(256), 0, s, part_val, part_idx, n, out);
  return hipGetLastError();
}

}  // namespace akvs
