// Reuse-specific kernels: check-layer divergence, probe selection, per-unit offsets,
// the fused re-rotation + dequantisation + weighted correction, and the cache quantiser.
#include "kernels.h"

namespace akvs {

// Rotate 8 lo/hi pairs (dims e0+i and e0+i+hd/2) by the angles of table row `p`.
__device__ __forceinline__ void rotate8(const float2 *rope_row, int e0, float (&lo)[8],
                                        float (&hi)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float2 cs = rope_row[e0 + i];
    const float a = lo[i], b = hi[i];
    lo[i] = a * cs.x - b * cs.y;
    hi[i] = b * cs.x + a * cs.y;
  }
}

template <typename T>
__host__ __device__ __forceinline__ const T *as(const void *p) {
  return reinterpret_cast<const T *>(p);
}

// ---------------------------------------------------------------------------------------
// Divergence: one wave per token. Work unit = (head, 8 lo/hi pairs) = 16 elements.
template <typename TF>
__global__ void k_divergence(const TF *k_fresh, const TF *v_fresh, CacheLayer cache, int n_tokens,
                             int hkv, int hd, const int32_t *tok_delta, const float2 *rope,
                             int rope_rows, float *d_k, float *d_v) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (t >= n_tokens) return;
  const int half = hd >> 1;
  const int units_per_head = half >> 3;
  const int units = hkv * units_per_head;
  int delta = tok_delta ? tok_delta[t] : 0;
  const bool bad = delta < 0 || delta >= rope_rows;
  if (bad) delta = 0;
  const float2 *rrow = rope + (size_t)delta * half;
  float sk = 0.f, sv = 0.f;
  for (int u = lane; u < units; u += 64) {
    const int h = u / units_per_head;
    const int e0 = (u - h * units_per_head) * 8;
    const size_t row = (size_t)t * hkv + h;
    float flo[8], fhi[8], clo[8], chi[8];
    // K
    load8(k_fresh + row * hd + e0, flo);
    load8(k_fresh + row * hd + e0 + half, fhi);
    cache_load8(cache.k, cache.k_meta, cache.dtype, row, hd, e0, clo);
    cache_load8(cache.k, cache.k_meta, cache.dtype, row, hd, e0 + half, chi);
    if (tok_delta) rotate8(rrow, e0, clo, chi);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float a = flo[i] - clo[i], b = fhi[i] - chi[i];
      sk = fmaf(a, a, sk);
      sk = fmaf(b, b, sk);
    }
    // V
    load8(v_fresh + row * hd + e0, flo);
    load8(v_fresh + row * hd + e0 + half, fhi);
    cache_load8(cache.v, cache.v_meta, cache.dtype, row, hd, e0, clo);
    cache_load8(cache.v, cache.v_meta, cache.dtype, row, hd, e0 + half, chi);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float a = flo[i] - clo[i], b = fhi[i] - chi[i];
      sv = fmaf(a, a, sv);
      sv = fmaf(b, b, sv);
    }
  }
  sk = wave_sum(sk);
  sv = wave_sum(sv);
  if (lane == 0) {
    d_k[t] = bad ? __builtin_nanf("") : sqrtf(sk);
    d_v[t] = bad ? __builtin_nanf("") : sqrtf(sv);
  }
}

hipError_t launch_divergence(const void *k_fresh, const void *v_fresh, int fresh_dtype,
                             CacheLayer cache, int n_tokens, int hkv, int hd,
                             const int32_t *tok_delta, const float *rope, int rope_rows,
                             float *d_k, float *d_v, hipStream_t s) {
  if (n_tokens == 0) return hipSuccess;
  dim3 g((n_tokens + 3) / 4), b(256);
  const float2 *r = reinterpret_cast<const float2 *>(rope);
  if (fresh_dtype == AKVS_BF16)
    hipLaunchKernelGGL(k_divergence<bf16_t>, g, b, 0, s, as<bf16_t>(k_fresh), as<bf16_t>(v_fresh),
                       cache, n_tokens, hkv, hd, tok_delta, r, rope_rows, d_k, d_v);
  else
    hipLaunchKernelGGL(k_divergence<float>, g, b, 0, s, as<float>(k_fresh), as<float>(v_fresh),
                       cache, n_tokens, hkv, hd, tok_delta, r, rope_rows, d_k, d_v);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Selection, pass 1: one block per unit. rank(j) = #{t : d_t > d_j or (d_t == d_j, t < j)};
// j is a probe iff rank(j) < b. Then the probe lists (ascending) are compacted by wave 0.
constexpr int SEL_TILE = 1024;

__global__ void k_select_rank(const float *d_k, const float *d_v, const int4 *meta, uint32_t flags,
                              int32_t *probe_k, int32_t *probe_v, float *w_k, float *w_v,
                              uint8_t *tok_flags, int32_t *chunk_rows) {
  __shared__ float sk[SEL_TILE], sv[SEL_TILE];
  const int c = blockIdx.x;
  const int4 mc = meta[c];  // (start, len, budget, csr offset)
  const int s0 = mc.x, n = mc.y, b = mc.z, off = mc.w;
  const bool given = (flags & AKVS_F_GIVEN_PROBES) != 0;
  const bool unit_w = (flags & AKVS_F_UNIT_WEIGHTS) != 0;
  // each thread keeps the ranks of up to 8 of its tokens in registers (n <= 8*blockDim)
  for (int jb = 0; jb < n; jb += 8 * blockDim.x) {
    int rk[8], rv[8];
    float dk[8], dv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = jb + u * blockDim.x + threadIdx.x;
      rk[u] = rv[u] = 0;
      dk[u] = (j < n && b > 0) ? d_k[s0 + j] : 0.f;
      dv[u] = (j < n && b > 0) ? d_v[s0 + j] : 0.f;
      // a NaN divergence ranks below every number (keeps exactly b probes per side)
      if (dk[u] != dk[u]) dk[u] = -INFINITY;
      if (dv[u] != dv[u]) dv[u] = -INFINITY;
    }
    if (!given && b > 0) {
      for (int tb = 0; tb < n; tb += SEL_TILE) {
        __syncthreads();
        for (int t = threadIdx.x; t < SEL_TILE && tb + t < n; t += blockDim.x) {
          const float a = d_k[s0 + tb + t], bv = d_v[s0 + tb + t];
          sk[t] = (a != a) ? -INFINITY : a;
          sv[t] = (bv != bv) ? -INFINITY : bv;
        }
        __syncthreads();
        const int tn = min(SEL_TILE, n - tb);
        for (int t = 0; t < tn; ++t) {
          const float a = sk[t], bv = sv[t];
          const int tt = tb + t;
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int j = jb + u * blockDim.x + threadIdx.x;
            rk[u] += (a > dk[u]) || (a == dk[u] && tt < j);
            rv[u] += (bv > dv[u]) || (bv == dv[u] && tt < j);
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = jb + u * blockDim.x + threadIdx.x;
      if (j >= n) continue;
      uint8_t f;
      if (given) {
        f = 0;
        for (int k = 0; k < b; ++k) {
          f |= (probe_k[off + k] == s0 + j) ? 1 : 0;
          f |= (probe_v[off + k] == s0 + j) ? 2 : 0;
        }
      } else {
        f = (uint8_t)((rk[u] < b ? 1 : 0) | (rv[u] < b ? 2 : 0));
      }
      tok_flags[s0 + j] = f;
      // w only multiplies the unit's offset, which is 0 when b == 0
      w_k[s0 + j] = b == 0 ? 0.f : (unit_w ? 1.f : fmaxf(fminf(dk[u], 1.f), 0.f));
      w_v[s0 + j] = b == 0 ? 0.f : (unit_w ? 1.f : fmaxf(fminf(dv[u], 1.f), 0.f));
    }
  }
  __syncthreads();
  if (threadIdx.x >= 64) return;
  // wave 0: ascending compaction of the probe lists and the union count
  const int lane = threadIdx.x;
  int ck = 0, cv = 0, cu = 0;
  for (int jb = 0; jb < n; jb += 64) {
    const int j = jb + lane;
    const uint8_t f = j < n ? tok_flags[s0 + j] : 0;
    const uint64_t mk = __ballot((f & 1) != 0);
    const uint64_t mv = __ballot((f & 2) != 0);
    const uint64_t mu = __ballot(f != 0);
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    if (!given) {
      if ((f & 1) && ck + __popcll(mk & below) < b) probe_k[off + ck + __popcll(mk & below)] = s0 + j;
      if ((f & 2) && cv + __popcll(mv & below) < b) probe_v[off + cv + __popcll(mv & below)] = s0 + j;
    }
    ck += __popcll(mk);
    cv += __popcll(mv);
    cu += __popcll(mu);
  }
  if (lane == 0) chunk_rows[c] = cu;
}

// Selection, pass 2: block i < m writes unit i's recomputed rows at its offset in R; block m
// writes the query rows and |R|.
__global__ void k_select_rows(const int4 *meta, int n_chunks, int t_ctx, int q,
                              const uint8_t *tok_flags, const int32_t *chunk_rows, int32_t *rows,
                              int32_t *n_rows, int32_t *fresh_row) {
  const int c = blockIdx.x;
  const int lane = threadIdx.x;  // one wave
  int base = 0;
  for (int i = lane; i < c; i += 64) base += chunk_rows[i];
  for (int o = 32; o > 0; o >>= 1) base += __shfl_xor(base, o, 64);
  if (c == n_chunks) {
    for (int t = lane; t < q; t += 64) {
      rows[base + t] = t_ctx + t;
      fresh_row[t_ctx + t] = base + t;
    }
    if (lane == 0) *n_rows = base + q;
    return;
  }
  const int4 mc = meta[c];
  int cnt = 0;
  for (int jb = 0; jb < mc.y; jb += 64) {
    const int j = jb + lane;
    const uint8_t f = j < mc.y ? tok_flags[mc.x + j] : 0;
    const uint64_t m = __ballot(f != 0);
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    if (j < mc.y) {
      if (f) {
        const int r = base + cnt + __popcll(m & below);
        rows[r] = mc.x + j;
        fresh_row[mc.x + j] = r;
      } else {
        fresh_row[mc.x + j] = -1;
      }
    }
    cnt += __popcll(m);
  }
}

hipError_t launch_select(const float *d_k, const float *d_v, const int32_t *meta, int n_chunks,
                         int t_ctx, int q, uint32_t flags, int32_t *probe_k, int32_t *probe_v,
                         float *w_k, float *w_v, uint8_t *tok_flags, int32_t *chunk_rows,
                         int32_t *rows, int32_t *n_rows, int32_t *fresh_row, hipStream_t s) {
  const int4 *m4 = reinterpret_cast<const int4 *>(meta);
  hipLaunchKernelGGL(k_select_rank, dim3(n_chunks), dim3(256), 0, s, d_k, d_v, m4, flags, probe_k,
                     probe_v, w_k, w_v, tok_flags, chunk_rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_select_rows, dim3(n_chunks + 1), dim3(64), 0, s, m4, n_chunks, t_ctx, q,
                     tok_flags, chunk_rows, rows, n_rows, fresh_row);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Per-unit offsets. grid = (m, 2 sides, pair blocks of 64); block = 4 waves. The unit's
// probe positions and their rows in the fresh buffers are first staged in LDS, so the
// data loads that follow are independent. Lane = one lo/hi pair of one head; wave w sums
// the probes k = w, w+4, ... in ascending order, and the four partial sums are added in
// wave order: a fixed fp32 summation order.
constexpr int OFF_MAXB = 1024;  // probes staged per pass

template <typename TF>
__global__ __launch_bounds__(256) void k_chunk_offset(const TF *k_fresh, const TF *v_fresh,
                                                      const int32_t *fresh_row, CacheLayer cache,
                                                      const int4 *meta, const int32_t *probe_k,
                                                      const int32_t *probe_v, uint32_t flags,
                                                      int hkv, int hd, const float2 *rope,
                                                      int rope_rows, float *mu_k, float *mu_v) {
  __shared__ int s_tok[OFF_MAXB], s_row[OFF_MAXB];
  __shared__ float s_part[4][64][2];
  const int c = blockIdx.x;
  const int side = blockIdx.y;  // 0 = K, 1 = V
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = hd >> 1;
  const int pairs = hkv * half;
  const int p = blockIdx.z * 64 + lane;
  const bool active = p < pairs;
  const int h = active ? p / half : 0, e = active ? p - h * half : 0;
  const int kvw = hkv * hd;
  const int4 mc = meta[c];
  const int b = mc.z;
  float *mu = (side == 0 ? mu_k : mu_v) + (size_t)c * kvw + h * hd;
  if (b == 0 || (flags & AKVS_F_NO_CORRECTION)) {
    if (active && wave == 0) {
      mu[e] = 0.f;
      mu[e + half] = 0.f;
    }
    return;
  }
  const TF *fresh = side == 0 ? k_fresh : v_fresh;
  const void *cb = side == 0 ? cache.k : cache.v;
  const _Float16 *cm = side == 0 ? cache.k_meta : cache.v_meta;
  const int32_t *probes = (side == 0 ? probe_k : probe_v) + mc.w;
  const int delta = (mc.x >= 0 && mc.x < rope_rows) ? mc.x : 0;
  const float2 cs = rope[(size_t)delta * half + e];
  float slo = 0.f, shi = 0.f;
  for (int kb = 0; kb < b; kb += OFF_MAXB) {
    const int nb = min(OFF_MAXB, b - kb);
    __syncthreads();
    for (int k = threadIdx.x; k < nb; k += blockDim.x) {
      const int j = probes[kb + k];
      const bool inside = j >= mc.x && j < mc.x + mc.y;  // a token of this unit
      const int r = inside ? fresh_row[j] : -1;
      s_tok[k] = inside ? j : -1;
      s_row[k] = r;
    }
    __syncthreads();
    if (active) {
      for (int k = wave; k < nb; k += 4) {
        const int j = s_tok[k], r = s_row[k];
        if (j < 0 || r < 0) continue;
        const size_t frow = (size_t)r * hkv + h;
        const size_t crow = (size_t)j * hkv + h;
        const float flo = load1(fresh + frow * hd + e), fhi = load1(fresh + frow * hd + e + half);
        float clo = cache_load1(cb, cm, cache.dtype, crow, hd, e);
        float chi = cache_load1(cb, cm, cache.dtype, crow, hd, e + half);
        if (side == 0) {
          const float a = clo, bb = chi;
          clo = a * cs.x - bb * cs.y;
          chi = bb * cs.x + a * cs.y;
        }
        slo += flo - clo;
        shi += fhi - chi;
      }
    }
  }
  s_part[wave][lane][0] = slo;
  s_part[wave][lane][1] = shi;
  __syncthreads();
  if (wave == 0 && active) {
    const float tlo = ((s_part[0][lane][0] + s_part[1][lane][0]) + s_part[2][lane][0]) + s_part[3][lane][0];
    const float thi = ((s_part[0][lane][1] + s_part[1][lane][1]) + s_part[2][lane][1]) + s_part[3][lane][1];
    mu[e] = tlo / (float)b;
    mu[e + half] = thi / (float)b;
  }
}

hipError_t launch_chunk_offset(const void *k_fresh, const void *v_fresh, int fresh_dtype,
                               const int32_t *fresh_row, CacheLayer cache, const int32_t *meta,
                               int n_chunks, const int32_t *probe_k, const int32_t *probe_v,
                               uint32_t flags, int hkv, int hd, const float *rope, int rope_rows,
                               float *mu_k, float *mu_v, hipStream_t s) {
  const int pairs = hkv * hd / 2;
  dim3 g(n_chunks, 2, (pairs + 63) / 64), b(256);
  const int4 *m4 = reinterpret_cast<const int4 *>(meta);
  const float2 *r = reinterpret_cast<const float2 *>(rope);
  if (fresh_dtype == AKVS_BF16)
    hipLaunchKernelGGL(k_chunk_offset<bf16_t>, g, b, 0, s, as<bf16_t>(k_fresh), as<bf16_t>(v_fresh),
                       fresh_row, cache, m4, probe_k, probe_v, flags, hkv, hd, r, rope_rows, mu_k,
                       mu_v);
  else
    hipLaunchKernelGGL(k_chunk_offset<float>, g, b, 0, s, as<float>(k_fresh), as<float>(v_fresh),
                       fresh_row, cache, m4, probe_k, probe_v, flags, hkv, hd, r, rope_rows, mu_k,
                       mu_v);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Fused re-rotation + dequantisation + weighted correction (+ fresh rows), K and V.
// Thread = (position t, head h, 8 lo/hi pairs). t < t_ctx: unit token; else query row.
// Unit holding context position t: the last i with meta[i].start <= t.
__device__ __forceinline__ int find_chunk(const int4 *meta, int n_chunks, int t) {
  int lo = 0, hi = n_chunks - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (meta[mid].x <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

template <typename TS>
__global__ void k_correction(CacheLayer cache, const float *mu_k, const float *mu_v,
                             const float *w_k, const float *w_v, const uint8_t *tok_flags,
                             const TS *k_fresh, const TS *v_fresh, const int32_t *fresh_row,
                             const int32_t *tok_chunk, const int32_t *tok_delta,
                             const int4 *meta, int n_chunks, int t_ctx,
                             int t_all, int hkv, int hd, uint32_t flags, const float2 *rope,
                             int rope_rows, TS *k_corr, TS *v_corr) {
  const int half = hd >> 1;
  const int units_per_head = half >> 3;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long per_tok = (long long)hkv * units_per_head;
  const int t = (int)(gid / per_tok);
  if (t >= t_all) return;
  const int rem = (int)(gid - (long long)t * per_tok);
  const int h = rem / units_per_head;
  const int e0 = (rem - h * units_per_head) * 8;
  const size_t orow = (size_t)t * hkv + h;
  TS *ko = k_corr + orow * hd;
  TS *vo = v_corr + orow * hd;
  const uint8_t f = (t < t_ctx) ? (tok_flags ? tok_flags[t] : 0) : 3;
  int chunk = 0, delta = 0;
  if (t < t_ctx) {
    if (tok_chunk) {
      chunk = tok_chunk[t];
      delta = tok_delta[t];
    } else if (meta) {
      chunk = find_chunk(meta, n_chunks, t);
      delta = meta[chunk].x;
    } else {
      delta = tok_delta[t];
    }
    if (delta < 0 || delta >= rope_rows) delta = 0;
    if (chunk < 0 || chunk >= n_chunks) chunk = 0;
  }
  const bool any = f != 0 && (flags & AKVS_F_FRESH_IF_RECOMPUTED);
  const bool fresh_k = (f & 1) || any;
  const bool fresh_v = (f & 2) || any;
  const int fr = (fresh_k || fresh_v) ? fresh_row[t] : -1;
  float lo[8], hi[8];
  // ---- K
  if (fresh_k) {
    if (fr >= 0) {
      const TS *src = k_fresh + ((size_t)fr * hkv + h) * hd;
      load8(src + e0, lo);
      load8(src + e0 + half, hi);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) lo[i] = hi[i] = 0.f;
    }
  } else {
    cache_load8(cache.k, cache.k_meta, cache.dtype, orow, hd, e0, lo);
    cache_load8(cache.k, cache.k_meta, cache.dtype, orow, hd, e0 + half, hi);
    rotate8(rope + (size_t)delta * half, e0, lo, hi);
    if (mu_k) {
      const float w = w_k[t];
      const float *mu = mu_k + (size_t)chunk * hkv * hd + h * hd;
      float ml[8], mh[8];
      load8(mu + e0, ml);
      load8(mu + e0 + half, mh);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        lo[i] = fmaf(w, ml[i], lo[i]);
        hi[i] = fmaf(w, mh[i], hi[i]);
      }
    }
  }
  store8(ko + e0, lo);
  store8(ko + e0 + half, hi);
  // ---- V
  if (fresh_v) {
    if (fr >= 0) {
      const TS *src = v_fresh + ((size_t)fr * hkv + h) * hd;
      load8(src + e0, lo);
      load8(src + e0 + half, hi);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) lo[i] = hi[i] = 0.f;
    }
  } else {
    cache_load8(cache.v, cache.v_meta, cache.dtype, orow, hd, e0, lo);
    cache_load8(cache.v, cache.v_meta, cache.dtype, orow, hd, e0 + half, hi);
    if (mu_v) {
      const float w = w_v[t];
      const float *mu = mu_v + (size_t)chunk * hkv * hd + h * hd;
      float ml[8], mh[8];
      load8(mu + e0, ml);
      load8(mu + e0 + half, mh);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        lo[i] = fmaf(w, ml[i], lo[i]);
        hi[i] = fmaf(w, mh[i], hi[i]);
      }
    }
  }
  store8(vo + e0, lo);
  store8(vo + e0 + half, hi);
}

hipError_t launch_correction(CacheLayer cache, const float *mu_k, const float *mu_v,
                             const float *w_k, const float *w_v, const uint8_t *tok_flags,
                             const void *k_fresh, const void *v_fresh, const int32_t *fresh_row,
                             const int32_t *tok_chunk, const int32_t *tok_delta,
                             const int32_t *meta, int n_chunks, int t_ctx,
                             int t_all, int hkv, int hd, uint32_t flags, const float *rope,
                             int rope_rows, void *k_corr, void *v_corr, int out_dtype,
                             hipStream_t s) {
  const int4 *m4 = reinterpret_cast<const int4 *>(meta);
  const long long threads = (long long)t_all * hkv * (hd / 16);
  if (threads == 0) return hipSuccess;
  dim3 g((unsigned)((threads + 255) / 256)), b(256);
  const float2 *r = reinterpret_cast<const float2 *>(rope);
  if (out_dtype == AKVS_BF16)
    hipLaunchKernelGGL(k_correction<bf16_t>, g, b, 0, s, cache, mu_k, mu_v, w_k, w_v, tok_flags,
                       as<bf16_t>(k_fresh), as<bf16_t>(v_fresh), fresh_row, tok_chunk, tok_delta,
                       m4, n_chunks, t_ctx, t_all, hkv, hd, flags, r, rope_rows,
                       reinterpret_cast<bf16_t *>(k_corr), reinterpret_cast<bf16_t *>(v_corr));
  else
    hipLaunchKernelGGL(k_correction<float>, g, b, 0, s, cache, mu_k, mu_v, w_k, w_v, tok_flags,
                       as<float>(k_fresh), as<float>(v_fresh), fresh_row, tok_chunk, tok_delta,
                       m4, n_chunks, t_ctx, t_all, hkv, hd, flags, r, rope_rows,
                       reinterpret_cast<float *>(k_corr), reinterpret_cast<float *>(v_corr));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Quantiser: one wave per (row, group of 64); lane = element.
template <typename TX>
__global__ void k_quantize(const TX *x, int n_rows, int hd, int bits, uint8_t *codes,
                           _Float16 *meta) {
  const int lane = threadIdx.x & 63;
  const int groups = hd / 64;
  const long long gid = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (gid >= (long long)n_rows * groups) return;
  const long long row = gid / groups;
  const int grp = (int)(gid - row * groups);
  const float v = load1(x + row * hd + grp * 64 + lane);
  const float mn = wave_min(v), mx = wave_max(v);
  const float levels = (float)((1 << bits) - 1);
  const _Float16 z16 = (_Float16)mn;
  const _Float16 s16 = (_Float16)__fdiv_rn(mx - mn, levels);
  const float zero = (float)z16, scale = (float)s16;
  int code = 0;
  if (scale != 0.f) {
    const float tq = rintf(__fdiv_rn(v - zero, scale));
    code = (int)fminf(fmaxf(tq, 0.f), levels);
  }
  const int per = 8 / bits;
  int packed = code << (bits * (lane % per));
  for (int o = 1; o < per; o <<= 1) packed |= __shfl_xor(packed, o, 64);
  if (lane % per == 0) codes[row * (hd * bits / 8) + grp * (64 * bits / 8) + lane / per] = (uint8_t)packed;
  if (lane == 0) {
    meta[2 * gid] = s16;
    meta[2 * gid + 1] = z16;
  }
}

hipError_t launch_quantize(const void *x, int x_dtype, int n_rows, int hd, int bits,
                           uint8_t *codes, _Float16 *meta, hipStream_t s) {
  const long long waves = (long long)n_rows * (hd / 64);
  if (waves == 0) return hipSuccess;
  dim3 g((unsigned)((waves + 3) / 4)), b(256);
  if (x_dtype == AKVS_BF16)
    hipLaunchKernelGGL(k_quantize<bf16_t>, g, b, 0, s, as<bf16_t>(x), n_rows, hd, bits, codes, meta);
  else
    hipLaunchKernelGGL(k_quantize<float>, g, b, 0, s, as<float>(x), n_rows, hd, bits, codes, meta);
  return hipGetLastError();
}

}  // namespace akvs
