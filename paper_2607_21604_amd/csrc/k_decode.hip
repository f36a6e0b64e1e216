// Decode-step kernels: the projections of one token as matrix-vector products (each
// weight row is read once, so these are HBM-bound) with the epilogues of the prefill
// GEMMs, and the greedy pick over the vocabulary logits.
//
// One wave owns one item: a pair of weight rows whose results an epilogue needs together
// (the two rotary halves of a q / k dimension, the gate and up rows of one SwiGLU unit, or
// two neighbouring rows). Lanes stride the reduction axis by 8 elements, several 16-byte
// loads in flight per lane; the wave sum uses a fixed butterfly, so results are
// reproducible bit for bit.
#include <algorithm>
#include <type_traits>

#include "kernels.h"

namespace akvs {

namespace {

// the prefill GEMMs' SiLU (hardware reciprocal in place of an IEEE division)
__device__ __forceinline__ float silu_dec(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
}

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

// NORM with bf16 weights: the first PRE 16-byte chunks of both rows of a lane are requested
// before the block normalises x, and consumed after it in the same k order as dot2.
constexpr int GV_PRE = 8;
__device__ __forceinline__ void acc_bf16x8(const u32x4_t &w, const float *xv, float &a) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a = fmaf(__uint_as_float(w[i] << 16), xv[2 * i], a);
    a = fmaf(__uint_as_float(w[i] & 0xffff0000u), xv[2 * i + 1], a);
  }
}

template <typename TW, typename TX, bool NORM>
__global__ __launch_bounds__(256) void k_gemv(const TX *__restrict__ x,
                                              const TW *__restrict__ W, int N, int K,
                                              GemvEpi e) {
  __shared__ float s_val[4];
  __shared__ int s_idx[4];
  extern __shared__ float s_x[];  // NORM: the normalised row [K]
  constexpr bool PREF = NORM && std::is_same<TW, bf16_t>::value;
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
  if (PREF) {
    constexpr int STRIDE = 64 * 8;
    const bf16_t *w0 = reinterpret_cast<const bf16_t *>(W) + (size_t)r0 * K;
    const bf16_t *w1 = reinterpret_cast<const bf16_t *>(W) + (size_t)r1 * K;
    u32x4_t p0[GV_PRE], p1[GV_PRE];
    if (live) {
#pragma unroll
      for (int p = 0; p < GV_PRE; ++p) {
        const int k = lane * 8 + p * STRIDE;
        if (k < K) {
          p0[p] = *reinterpret_cast<const u32x4_t *>(w0 + k);
          p1[p] = *reinterpret_cast<const u32x4_t *>(w1 + k);
        }
      }
    }
    norm_row_lds(reinterpret_cast<const float *>(x), reinterpret_cast<const bf16_t *>(e.norm), K,
                 e.eps, s_x);
    if (live) {
      float a0 = 0.f, a1 = 0.f;
#pragma unroll
      for (int p = 0; p < GV_PRE; ++p) {
        const int k = lane * 8 + p * STRIDE;
        if (k < K) {
          float xv[8];
          load8(s_x + k, xv);
          acc_bf16x8(p0[p], xv, a0);
          acc_bf16x8(p1[p], xv, a1);
        }
      }
      for (int k = lane * 8 + GV_PRE * STRIDE; k < K; k += STRIDE) {
        float xv[8], wa[8], wb[8];
        load8(s_x + k, xv);
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
  } else {
    if (NORM)
      norm_row_lds(reinterpret_cast<const float *>(x), reinterpret_cast<const TW *>(e.norm), K,
                   e.eps, s_x);
    if (live) {
      if (NORM)
        dot2(W + (size_t)r0 * K, W + (size_t)r1 * K, static_cast<const float *>(s_x), K, lane,
             s0, s1);
      else
        dot2(W + (size_t)r0 * K, W + (size_t)r1 * K, x, K, lane, s0, s1);
    }
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


// ---- attention of the one new row ------------------------------------------------------
// Block = (KV head, chunk of <= DA_MAX_KEYS keys), 256 threads, all G query heads of that KV
// head, so every key / value byte is read once; every thread issues all of its K and V loads
// first. Keys: thread t holds dims (t % L) * 8 ..+7 of keys t / L + j * KPI (L = hd / 8),
// so a score is a sum over the L lanes of one row. Values: thread t holds dims
// ((t / 16) % L) * 8 ..+7 of keys 16 (t / (16 L)) + t % 16 + j * KPI, so p * v is summed
// over the 16 lanes of one row. Both sums use DPP lane moves inside a 16-lane row (no LDS
// round trip). One wave per head forms the chunk's maximum m, p = 2^(s - m) and l = sum p.
// The chunk's (o, m, l) go to the partial buffers; k_attn_decode_merge combines the chunks.
// Fixed orders throughout.
constexpr int DA_MAX_KEYS = 128, DA_MAXG = 8;

// x + (x of the lane given by a DPP control inside each 16-lane row)
template <int CTRL>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
// Sum over aligned groups of N lanes (N = 8 or 16) inside a row: pairs, quads, then the
// mirrored half rows and rows; every lane of a group ends with the group's sum.
template <int N>
__device__ __forceinline__ float row_sum(float x) {
  x = dpp_add<0xB1>(x);   // quad_perm [1,0,3,2]: lane ^ 1
  x = dpp_add<0x4E>(x);   // quad_perm [2,3,0,1]: lane ^ 2
  x = dpp_add<0x141>(x);  // row_half_mirror: quad 0 <-> quad 1 of each 8 lanes
  if (N == 16) x = dpp_add<0x140>(x);  // row_mirror: the two halves of the row
  return x;
}

template <int HD>
__global__ __launch_bounds__(256) void k_attn_decode(const bf16_t *__restrict__ q,
                                                     const bf16_t *__restrict__ Kc,
                                                     const bf16_t *__restrict__ Vc, int n_keys,
                                                     int hkv, int G, int chunk,
                                                     float scale_log2, float *__restrict__ part_o,
                                                     float *__restrict__ part_ml) {
  constexpr int L = HD / 8, KPI = 256 / L, NIT = DA_MAX_KEYS / KPI, VS = 256 / (16 * L);
  __shared__ float s_p[DA_MAXG][DA_MAX_KEYS];
  __shared__ float s_m[DA_MAXG], s_l[DA_MAXG];
  __shared__ float s_o[VS][DA_MAXG][HD];
  const int kvh = blockIdx.x % hkv, c = blockIdx.x / hkv;
  const int c0 = c * chunk, nk = min(chunk, n_keys - c0);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int li = t % L, ks = t / L;                                 // key-side map
  const int kg = t & 15, dc = (t >> 4) % L, vs = t / (16 * L);      // value-side map
  u32x4_t kr[NIT], vr[NIT];
#pragma unroll
  for (int j = 0; j < NIT; ++j) {
    if (j * KPI < nk) {  // rows past the chunk re-read its last key
      const int kk = min(ks + j * KPI, nk - 1), vk = min(vs * 16 + kg + j * KPI, nk - 1);
      kr[j] = *reinterpret_cast<const u32x4_t *>(Kc + ((size_t)(c0 + kk) * hkv + kvh) * HD + li * 8);
      vr[j] = *reinterpret_cast<const u32x4_t *>(Vc + ((size_t)(c0 + vk) * hkv + kvh) * HD + dc * 8);
    }
  }
#pragma unroll
  for (int g = 0; g < DA_MAXG; ++g) {
    if (g >= G) break;
    float qv[8];
    load8(q + (size_t)(kvh * G + g) * HD + li * 8, qv);
#pragma unroll
    for (int j = 0; j < NIT; ++j) {
      if (j * KPI >= nk) break;
      float d = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        d = fmaf(qv[2 * i], __uint_as_float(kr[j][i] << 16), d);
        d = fmaf(qv[2 * i + 1], __uint_as_float(kr[j][i] & 0xffff0000u), d);
      }
      d = row_sum<L>(d);
      const int kk = ks + j * KPI;
      if (li == 0 && kk < nk) s_p[g][kk] = d * scale_log2;
    }
  }
  __syncthreads();
  for (int g = wave; g < G; g += 4) {
    float mx = -INFINITY;
    for (int k = lane; k < nk; k += 64) mx = fmaxf(mx, s_p[g][k]);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int k = lane; k < nk; k += 64) {
      const float p = __builtin_amdgcn_exp2f(s_p[g][k] - mx);
      s_p[g][k] = p;
      sum += p;
    }
    sum = wave_sum(sum);
    if (lane == 0) {
      s_m[g] = mx;
      s_l[g] = sum;
    }
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < DA_MAXG; ++g) {
    if (g >= G) break;
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
#pragma unroll
    for (int j = 0; j < NIT; ++j) {
      if (j * KPI >= nk) break;
      const int vk = vs * 16 + kg + j * KPI;
      const float p = vk < nk ? s_p[g][vk] : 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] = fmaf(p, __uint_as_float(vr[j][i] << 16), acc[2 * i]);
        acc[2 * i + 1] = fmaf(p, __uint_as_float(vr[j][i] & 0xffff0000u), acc[2 * i + 1]);
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = row_sum<16>(acc[i]);
    if (kg == 0) {
#pragma unroll
      for (int i = 0; i < 8; ++i) s_o[vs][g][dc * 8 + i] = acc[i];
    }
  }
  __syncthreads();
  for (int e = t; e < G * HD; e += 256) {
    const int g = e / HD, d = e - g * HD;
    float o = s_o[0][g][d];
#pragma unroll
    for (int v = 1; v < VS; ++v) o += s_o[v][g][d];
    const size_t i = (size_t)c * hkv * G + kvh * G + g;
    part_o[i * HD + d] = o;
    if (d == 0) {
      part_ml[2 * i] = s_m[g];
      part_ml[2 * i + 1] = s_l[g];
    }
  }
}

// out[h][d] = sum_c 2^(m_c - M) o_c[h][d] / sum_c 2^(m_c - M) l_c, M = max_c m_c, chunks
// added in index order. Block = (head, 32 head dims), thread = one dim of chunks
// cg, cg + 8, ...; the eight chunk groups are added in order through LDS.
__global__ __launch_bounds__(256) void k_attn_decode_merge(const float *__restrict__ part_o,
                                                           const float *__restrict__ part_ml,
                                                           int n_chunks, int hq, int hd,
                                                           bf16_t *__restrict__ out) {
  __shared__ float s_red[8][33];
  __shared__ float s_lr[8], s_mx[4];
  const int per_head = hd / 32;
  const int h = blockIdx.x / per_head, d0 = (blockIdx.x % per_head) * 32;
  const int t = threadIdx.x, d = t & 31, cg = t >> 5;
  float mx = -INFINITY;
  for (int c = t; c < n_chunks; c += 256) mx = fmaxf(mx, part_ml[2 * ((size_t)c * hq + h)]);
  mx = wave_max(mx);
  if ((t & 63) == 0) s_mx[t >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(s_mx[0], s_mx[1]), fmaxf(s_mx[2], s_mx[3]));
  float o = 0.f, l = 0.f;
  for (int c = cg; c < n_chunks; c += 8) {
    const size_t i = (size_t)c * hq + h;
    const float w = __builtin_amdgcn_exp2f(part_ml[2 * i] - mx);
    o = fmaf(w, part_o[i * hd + d0 + d], o);
    l = fmaf(w, part_ml[2 * i + 1], l);
  }
  s_red[cg][d] = o;
  if (d == 0) s_lr[cg] = l;
  __syncthreads();
  if (t < 32) {
    float so = 0.f, sl = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      so += s_red[k][t];
      sl += s_lr[k];
    }
    store1(out + (size_t)h * hd + d0 + t, so / sl);
  }
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

// Chunks of the one-row attention: about 512 blocks over the KV heads, chunks of at most
// DA_MAX_KEYS keys, a multiple of 16.
int decode_attn_chunks(int n_keys, int hkv, int *chunk_keys) {
  int per = (512 + hkv - 1) / hkv;
  int chunk = (n_keys + per - 1) / per;
  chunk = std::min(DA_MAX_KEYS, std::max(16, (chunk + 15) / 16 * 16));
  *chunk_keys = chunk;
  return (n_keys + chunk - 1) / chunk;
}

hipError_t launch_attention_decode(const void *q, const void *k, const void *v, int n_keys,
                                   int hq, int hkv, int hd, void *out, float *part_o,
                                   float *part_ml, hipStream_t s) {
  const int G = hq / hkv;
  if (n_keys < 1 || G < 1 || G > DA_MAXG || hq % hkv || (hd != 64 && hd != 128))
    return hipErrorInvalidValue;
  int chunk;
  const int n_chunks = decode_attn_chunks(n_keys, hkv, &chunk);
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
  const bf16_t *Q = reinterpret_cast<const bf16_t *>(q);
  const bf16_t *K = reinterpret_cast<const bf16_t *>(k);
  const bf16_t *V = reinterpret_cast<const bf16_t *>(v);
  if (hd == 128)
    hipLaunchKernelGGL(k_attn_decode<128>, dim3(n_chunks * hkv), dim3(256), 0, s, Q, K, V, n_keys,
                       hkv, G, chunk, scale_log2, part_o, part_ml);
  else
    hipLaunchKernelGGL(k_attn_decode<64>, dim3(n_chunks * hkv), dim3(256), 0, s, Q, K, V, n_keys,
                       hkv, G, chunk, scale_log2, part_o, part_ml);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_attn_decode_merge, dim3(hq * (hd / 32)), dim3(256), 0, s, part_o, part_ml,
                     n_chunks, hq, hd, reinterpret_cast<bf16_t *>(out));
  return hipGetLastError();
}

hipError_t launch_pick(const float *part_val, const int32_t *part_idx, int n, int32_t *out,
                       hipStream_t s) {
  hipLaunchKernelGGL(k_pick, dim3(1), dim3(256), 0, s, part_val, part_idx, n, out);
  return hipGetLastError();
}

}  // namespace akvs
