// Attention of (sparse, position-sorted) query rows over a causal key range.
//
// bf16 path: one block = 64 query rows x 1 query head, 4 waves of 16 rows. Keys stream
// through LDS in tiles of 64 (K row-major, V transposed). Scores are computed transposed,
// S^T = K Q^T, with MFMA 16x16x32 bf16: each lane then holds 16 scores of ONE query row,
// so the online softmax needs only two cross-lane steps, and the probabilities already
// sit in the operand layout of the second product O^T = V^T P^T (the pairing of the
// 32 contraction slots with keys is a fixed permutation applied to both operands).
// Row tiles are launched longest-first (rows are sorted by position, so later tiles
// see more keys).
#include "kernels.h"

namespace akvs {

template <int HD>
__global__ __launch_bounds__(256) void k_attn_bf16(const bf16_t *__restrict__ Q,
                                                   const int32_t *pos, int pos0, int rows,
                                                   const int32_t *rows_dev,
                                                   const bf16_t *__restrict__ Kc,
                                                   const bf16_t *__restrict__ Vc, int n_keys,
                                                   int hq, int hkv, float scale_log2,
                                                   bf16_t *__restrict__ out) {
  constexpr int KS = HD / 32;  // contraction steps of S
  constexpr int HB = HD / 16;  // 16-wide head-dim blocks of O
  constexpr int KST = HD + 8;  // K tile row stride (bf16)
  constexpr int VST = 64 + 8;  // V^T tile row stride (bf16)
  __shared__ __attribute__((aligned(16))) bf16_t Ks[64 * KST];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[HD * VST];
  __shared__ int s_max[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tile = gridDim.x - 1 - blockIdx.x;
  const int head = blockIdx.y;
  const int kvh = head / (hq / hkv);
  int R = rows;
  if (rows_dev) R = min(R, *rows_dev);
  const int row0 = tile * 64;
  if (row0 >= R) return;
  const int r = row0 + wave * 16 + (lane & 15);
  const bool rvalid = r < R;
  const int rp = rvalid ? (pos ? pos[r] : pos0 + r) : -1;
  int wmax = rp;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) wmax = max(wmax, __shfl_xor(wmax, o, 64));
  if (lane == 0) s_max[wave] = wmax;
  __syncthreads();
  const int bmax = max(max(s_max[0], s_max[1]), max(s_max[2], s_max[3]));
  const int kv_end = min(n_keys, bmax + 1);
  const int nkt = (kv_end + 63) / 64;
  const int rpos = rvalid ? rp : 0;

  bf16x8_t qf[KS];
  {
    const bf16_t *qrow = Q + ((size_t)(rvalid ? r : row0) * hq + head) * HD + (lane >> 4) * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8_t *>(qrow + ks * 32);
  }
  f32x4_t o[HB];
#pragma unroll
  for (int hb = 0; hb < HB; ++hb) o[hb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  for (int kt = 0; kt < nkt; ++kt) {
    const int key0 = kt * 64;
    __syncthreads();
    for (int c = threadIdx.x; c < 64 * HD / 8; c += 256) {
      const int kr = c / (HD / 8);
      const int e0 = (c - kr * (HD / 8)) * 8;
      const int key = key0 + kr;
      uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (key < kv_end) {
        const size_t off = ((size_t)key * hkv + kvh) * HD + e0;
        kv = *reinterpret_cast<const uint4 *>(Kc + off);
        vv = *reinterpret_cast<const uint4 *>(Vc + off);
      }
      *reinterpret_cast<uint4 *>(Ks + kr * KST + e0) = kv;
      const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        Vt[(e0 + 2 * i) * VST + kr] = (bf16_t)(w[i] & 0xffffu);
        Vt[(e0 + 2 * i + 1) * VST + kr] = (bf16_t)(w[i] >> 16);
      }
    }
    __syncthreads();
    if (key0 > wmax) continue;  // whole wave is before this key tile

    f32x4_t s[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      s[kb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
      const bf16_t *krow = Ks + (kb * 16 + (lane & 15)) * KST + (lane >> 4) * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t *>(krow + ks * 32);
        s[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[ks], s[kb], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = key0 + kb * 16 + (lane >> 4) * 4 + i;
        float v = s[kb][i] * scale_log2;
        if (key > rpos || key >= kv_end) v = -INFINITY;
        s[kb][i] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_run == -INFINITY) ? 0.f : exp2f(m_run - m_new);
    float rs = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = (s[kb][i] == -INFINITY) ? 0.f : exp2f(s[kb][i] - m_new);
        s[kb][i] = p;
        rs += p;
      }
    rs += __shfl_xor(rs, 16, 64);
    rs += __shfl_xor(rs, 32, 64);
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) o[hb] *= alpha;

#pragma unroll
    for (int t = 0; t < 2; ++t) {
      uint32_t pw[4];
      pw[0] = pack_bf2(s[2 * t][0], s[2 * t][1]);
      pw[1] = pack_bf2(s[2 * t][2], s[2 * t][3]);
      pw[2] = pack_bf2(s[2 * t + 1][0], s[2 * t + 1][1]);
      pw[3] = pack_bf2(s[2 * t + 1][2], s[2 * t + 1][3]);
      bf16x8_t pb;
      __builtin_memcpy(&pb, pw, 16);
#pragma unroll
      for (int hb = 0; hb < HB; ++hb) {
        const bf16_t *vrow = Vt + (hb * 16 + (lane & 15)) * VST + 32 * t + (lane >> 4) * 4;
        uint32_t vw[4];
        const uint2 x0 = *reinterpret_cast<const uint2 *>(vrow);
        const uint2 x1 = *reinterpret_cast<const uint2 *>(vrow + 16);
        vw[0] = x0.x; vw[1] = x0.y; vw[2] = x1.x; vw[3] = x1.y;
        bf16x8_t a;
        __builtin_memcpy(&a, vw, 16);
        o[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb, o[hb], 0, 0, 0);
      }
    }
  }
  if (!rvalid) return;
  const float inv = 1.0f / l_run;
  bf16_t *orow = out + ((size_t)r * hq + head) * HD + (lane >> 4) * 4;
#pragma unroll
  for (int hb = 0; hb < HB; ++hb)
    store4(orow + hb * 16, o[hb][0] * inv, o[hb][1] * inv, o[hb][2] * inv, o[hb][3] * inv);
}

// fp32 path (small models): one wave per (row, head), keys in tiles of 64, online softmax.
template <int HD>
__global__ __launch_bounds__(64) void k_attn_f32(const float *__restrict__ Q, const int32_t *pos,
                                                 int pos0, int rows, const int32_t *rows_dev,
                                                 const float *__restrict__ Kc,
                                                 const float *__restrict__ Vc, int n_keys, int hq,
                                                 int hkv, float scale, float *__restrict__ out) {
  constexpr int PER = HD / 64;
  __shared__ float qs[HD];
  __shared__ float ps[64];
  const int lane = threadIdx.x;
  const int r = blockIdx.x, head = blockIdx.y;
  int R = rows;
  if (rows_dev) R = min(R, *rows_dev);
  if (r >= R) return;
  const int kvh = head / (hq / hkv);
  const int rp = pos ? pos[r] : pos0 + r;
  const int kv_end = min(n_keys, rp + 1);
  const float *q = Q + ((size_t)r * hq + head) * HD;
  for (int e = lane; e < HD; e += 64) qs[e] = q[e];
  __syncthreads();
  float m = -INFINITY, l = 0.f, acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) acc[i] = 0.f;
  for (int key0 = 0; key0 < kv_end; key0 += 64) {
    const int key = key0 + lane;
    float sc = -INFINITY;
    if (key < kv_end) {
      const float *k = Kc + ((size_t)key * hkv + kvh) * HD;
      float d = 0.f;
      for (int e = 0; e < HD; ++e) d = fmaf(qs[e], k[e], d);
      sc = d * scale;
    }
    const float mx = wave_max(sc);
    const float m_new = fmaxf(m, mx);
    const float alpha = (m == -INFINITY) ? 0.f : __expf(m - m_new);
    const float p = (sc == -INFINITY) ? 0.f : __expf(sc - m_new);
    l = l * alpha + wave_sum(p);
    m = m_new;
    __syncthreads();
    ps[lane] = p;
    __syncthreads();
    const int nk = min(64, kv_end - key0);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = lane + 64 * i;
      float a = acc[i] * alpha;
      for (int j = 0; j < nk; ++j) a = fmaf(ps[j], Vc[((size_t)(key0 + j) * hkv + kvh) * HD + e], a);
      acc[i] = a;
    }
  }
  float *o = out + ((size_t)r * hq + head) * HD;
#pragma unroll
  for (int i = 0; i < PER; ++i) o[lane + 64 * i] = acc[i] / l;
}

hipError_t launch_attention(const void *q, const int32_t *pos, int pos0, int rows,
                            const int32_t *rows_dev, const void *k, const void *v, int n_keys,
                            int hq, int hkv, int hd, int dtype, void *out, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (dtype == AKVS_BF16) {
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    dim3 g((rows + 63) / 64, hq), b(256);
    const bf16_t *Q = reinterpret_cast<const bf16_t *>(q);
    const bf16_t *K = reinterpret_cast<const bf16_t *>(k);
    const bf16_t *V = reinterpret_cast<const bf16_t *>(v);
    bf16_t *O = reinterpret_cast<bf16_t *>(out);
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_bf16<128>, g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V, n_keys,
                         hq, hkv, scale_log2, O);
    else
      hipLaunchKernelGGL(k_attn_bf16<64>, g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V, n_keys,
                         hq, hkv, scale_log2, O);
  } else {
    const float scale = 1.0f / sqrtf((float)hd);
    dim3 g(rows, hq), b(64);
    const float *Q = reinterpret_cast<const float *>(q);
    const float *K = reinterpret_cast<const float *>(k);
    const float *V = reinterpret_cast<const float *>(v);
    float *O = reinterpret_cast<float *>(out);
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_f32<128>, g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V, n_keys,
                         hq, hkv, scale, O);
    else
      hipLaunchKernelGGL(k_attn_f32<64>, g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V, n_keys,
                         hq, hkv, scale, O);
  }
  return hipGetLastError();
}

}  // namespace akvs
