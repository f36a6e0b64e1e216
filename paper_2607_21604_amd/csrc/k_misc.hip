// Small bandwidth kernels: rotary table, embedding gather, RMSNorm, row gather.
#include "kernels.h"

namespace akvs {

// table[p][k] = (cos, sin)(p * theta^(-2k/hd)); angle and trig in fp64.
__global__ void k_rope_table(int p0, int n_pos, int half, int hd, double theta, float2 *table) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_pos * half) return;
  const int row = i / half, k = i - row * half;
  const int p = p0 + row;
  const double inv = pow(theta, (-2.0 * (double)k) / (double)hd);
  const double a = (double)p * inv;
  double sn, cs;
  sincos(a, &sn, &cs);
  table[i] = make_float2((float)cs, (float)sn);
}

hipError_t launch_rope_table(int p0, int n_pos, int head_dim, double theta, float *table,
                             hipStream_t s) {
  const int half = head_dim / 2;
  const int total = n_pos * half;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(k_rope_table, dim3((total + 255) / 256), dim3(256), 0, s, p0, n_pos, half,
                     head_dim, theta, reinterpret_cast<float2 *>(table));
  return hipGetLastError();
}

template <typename TE>
__global__ void k_embed(const int32_t *tok, int n, const TE *embed, int vocab, int D, float *h) {
  const int t = blockIdx.x;
  if (t >= n) return;
  const int id = tok[t];
  float *dst = h + (size_t)t * D;
  const bool ok = id >= 0 && id < vocab;
  const TE *src = embed + (size_t)(ok ? id : 0) * D;
  for (int e = threadIdx.x * 8; e < D; e += blockDim.x * 8) {
    float v[8];
    load8(src + e, v);
    if (!ok) {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = 0.f;
    }
    store8(dst + e, v);
  }
}

hipError_t launch_embed(const int32_t *tok, int n, const void *embed, int dtype, int vocab, int D,
                        float *h, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (dtype == AKVS_BF16)
    hipLaunchKernelGGL(k_embed<bf16_t>, dim3(n), dim3(128), 0, s, tok, n,
                       reinterpret_cast<const bf16_t *>(embed), vocab, D, h);
  else
    hipLaunchKernelGGL(k_embed<float>, dim3(n), dim3(128), 0, s, tok, n,
                       reinterpret_cast<const float *>(embed), vocab, D, h);
  return hipGetLastError();
}

// One block (256 threads) per row; D % 8 == 0. Sum of squares with a fixed reduction tree.
// Rows of up to RMS_REG * 2048 elements are read once into registers (row and gain loads
// all in flight before the sum); longer rows take a second pass over the row.
constexpr int RMS_REG = 4;
template <typename TG, typename TO>
__global__ void k_rmsnorm(const float *h, int ldh, int rows, const int32_t *rows_dev,
                          const int32_t *base_dev, const TG *gain, int D, float eps, TO *out,
                          int ldo) {
  const int i = blockIdx.x;
  int lim = rows;
  if (rows_dev && !base_dev) lim = min(lim, *rows_dev);
  if (i >= lim) return;
  int src = i;
  if (base_dev) {
    src = *base_dev - rows + i;
    if (src < 0) return;
  }
  const float *x = h + (size_t)src * ldh;
  __shared__ float red[4];
  TO *y = out + (size_t)i * ldo;
  if (D <= RMS_REG * 256 * 8) {  // one read of the row, kept in registers
    float v[RMS_REG][8], g[RMS_REG][8];
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < RMS_REG; ++c) {
      const int e = threadIdx.x * 8 + c * 256 * 8;
      if (e < D) {
        load8(x + e, v[c]);
        load8(gain + e, g[c]);
      }
    }
#pragma unroll
    for (int c = 0; c < RMS_REG; ++c) {
      if (threadIdx.x * 8 + c * 256 * 8 < D) {
#pragma unroll
        for (int k = 0; k < 8; ++k) ss = fmaf(v[c][k], v[c][k], ss);
      }
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float tot = (red[0] + red[1]) + (red[2] + red[3]);
    const float inv = 1.0f / sqrtf(tot / (float)D + eps);
#pragma unroll
    for (int c = 0; c < RMS_REG; ++c) {
      const int e = threadIdx.x * 8 + c * 256 * 8;
      if (e < D) {
#pragma unroll
        for (int k = 0; k < 8; ++k) v[c][k] = v[c][k] * inv * g[c][k];
        store8(y + e, v[c]);
      }
    }
    return;
  }
  float ss = 0.f;
  for (int e = threadIdx.x * 8; e < D; e += 256 * 8) {
    float v[8];
    load8(x + e, v);
#pragma unroll
    for (int k = 0; k < 8; ++k) ss = fmaf(v[k], v[k], ss);
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)D + eps);
  for (int e = threadIdx.x * 8; e < D; e += 256 * 8) {
    float v[8], g[8];
    load8(x + e, v);
    load8(gain + e, g);
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = v[k] * inv * g[k];
    store8(y + e, v);
  }
}

hipError_t launch_rmsnorm(const float *h, int ldh, int rows, const int32_t *rows_dev,
                          const int32_t *base_dev, const void *gain, int gain_dtype, int D,
                          float eps, void *out, int out_dtype, int ldo, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  dim3 g(rows), b(256);
  if (gain_dtype == AKVS_BF16) {
    const bf16_t *gn = reinterpret_cast<const bf16_t *>(gain);
    if (out_dtype == AKVS_BF16)
      hipLaunchKernelGGL((k_rmsnorm<bf16_t, bf16_t>), g, b, 0, s, h, ldh, rows, rows_dev, base_dev,
                         gn, D, eps, reinterpret_cast<bf16_t *>(out), ldo);
    else
      hipLaunchKernelGGL((k_rmsnorm<bf16_t, float>), g, b, 0, s, h, ldh, rows, rows_dev, base_dev,
                         gn, D, eps, reinterpret_cast<float *>(out), ldo);
  } else {
    const float *gn = reinterpret_cast<const float *>(gain);
    if (out_dtype == AKVS_BF16)
      hipLaunchKernelGGL((k_rmsnorm<float, bf16_t>), g, b, 0, s, h, ldh, rows, rows_dev, base_dev,
                         gn, D, eps, reinterpret_cast<bf16_t *>(out), ldo);
    else
      hipLaunchKernelGGL((k_rmsnorm<float, float>), g, b, 0, s, h, ldh, rows, rows_dev, base_dev,
                         gn, D, eps, reinterpret_cast<float *>(out), ldo);
  }
  return hipGetLastError();
}

__global__ void k_gather_rows(const float *src, int n_src, const int32_t *idx, int cap,
                              const int32_t *n_dev, int D, float *dst, const int32_t *dst_base) {
  const int i = blockIdx.x;
  if (i >= cap || i >= *n_dev) return;
  const int j = idx[i];
  const bool ok = j >= 0 && j < n_src;
  const float *a = src + (size_t)(ok ? j : 0) * D;
  float *b = dst + ((size_t)(dst_base ? *dst_base : 0) + i) * D;
  for (int e = threadIdx.x * 4; e < D; e += blockDim.x * 4)
    *reinterpret_cast<float4 *>(b + e) =
        ok ? *reinterpret_cast<const float4 *>(a + e) : make_float4(0.f, 0.f, 0.f, 0.f);
}

hipError_t launch_gather_rows(const float *src, int n_src, const int32_t *idx, int cap,
                              const int32_t *n_dev, int D, float *dst, hipStream_t s,
                              const int32_t *dst_base) {
  if (cap == 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_rows, dim3(cap), dim3(256), 0, s, src, n_src, idx, cap, n_dev, D,
                     dst, dst_base);
  return hipGetLastError();
}

// dst[i] = src[base + *n_dev - n + i] for i < n (rows of row_bytes bytes, a multiple of 16).
__global__ void k_copy_tail_rows(const char *src, size_t row_bytes, int n, const int32_t *n_dev,
                                 char *dst, const int32_t *src_base) {
  const int i = blockIdx.x;
  const int j = *n_dev - n + i;
  if (i >= n || j < 0) return;
  const size_t row = (size_t)(src_base ? *src_base : 0) + j;
  const uint4 *a = reinterpret_cast<const uint4 *>(src + row * row_bytes);
  uint4 *b = reinterpret_cast<uint4 *>(dst + (size_t)i * row_bytes);
  for (size_t e = threadIdx.x; e < row_bytes / 16; e += blockDim.x) b[e] = a[e];
}

hipError_t launch_copy_tail_rows(const void *src, size_t row_bytes, int n, const int32_t *n_dev,
                                 void *dst, hipStream_t s, const int32_t *src_base) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_tail_rows, dim3(n), dim3(256), 0, s,
                     reinterpret_cast<const char *>(src), row_bytes, n, n_dev,
                     reinterpret_cast<char *>(dst), src_base);
  return hipGetLastError();
}

// row_off[b] = n_rows[0] + ... + n_rows[b-1], b <= B (one thread: B is small).
__global__ void k_batch_layout(const int32_t *n_rows, int B, int32_t *row_off) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  int32_t acc = 0;
  for (int b = 0; b < B; ++b) {
    row_off[b] = acc;
    acc += n_rows[b];
  }
  row_off[B] = acc;
}

hipError_t launch_batch_layout(const int32_t *n_rows, int B, int32_t *row_off, hipStream_t s) {
  hipLaunchKernelGGL(k_batch_layout, dim3(1), dim3(64), 0, s, n_rows, B, row_off);
  return hipGetLastError();
}

// dst[*dst_base + i] = src[i], i < min(cap, *n_dev)
__global__ void k_copy_ints_at(const int32_t *src, int cap, const int32_t *n_dev, int32_t *dst,
                               const int32_t *dst_base) {
  const int n = min(cap, *n_dev);
  const int base = *dst_base;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    dst[base + i] = src[i];
}

hipError_t launch_copy_ints_at(const int32_t *src, int cap, const int32_t *n_dev, int32_t *dst,
                               const int32_t *dst_base, hipStream_t s) {
  if (cap == 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_ints_at, dim3((cap + 255) / 256), dim3(256), 0, s, src, cap, n_dev,
                     dst, dst_base);
  return hipGetLastError();
}

// one 32-bit value: dst[0] = src[0]
__global__ void k_copy_int(const int32_t *src, int32_t *dst) {
  if (blockIdx.x == 0 && threadIdx.x == 0) dst[0] = src[0];
}

hipError_t launch_copy_int(const int32_t *src, int32_t *dst, hipStream_t s) {
  hipLaunchKernelGGL(k_copy_int, dim3(1), dim3(64), 0, s, src, dst);
  return hipGetLastError();
}

__global__ void k_token_setup(const int4 *meta, int n_chunks, int32_t *tok_delta,
                              int32_t *tok_chunk) {
  const int c = blockIdx.x;
  if (c >= n_chunks) return;
  const int4 mc = meta[c];
  for (int j = threadIdx.x; j < mc.y; j += blockDim.x) {
    tok_delta[mc.x + j] = mc.x;
    tok_chunk[mc.x + j] = c;
  }
}

hipError_t launch_token_setup(const int32_t *meta, int n_chunks, int32_t *tok_delta,
                              int32_t *tok_chunk, hipStream_t s) {
  hipLaunchKernelGGL(k_token_setup, dim3(n_chunks), dim3(256), 0, s,
                     reinterpret_cast<const int4 *>(meta), n_chunks, tok_delta, tok_chunk);
  return hipGetLastError();
}

// ---- measurement helper --------------------------------------------------------------
// A loop of independent v_mfma_f32_32x32x16_bf16 (8 accumulators per wave, no other work)
// that keeps the matrix cores busy: the reference for the MFMA-busy counters and for the
// rate the chip sustains. The operands are random bf16 values in [-1, 1), four sets per
// lane used in turn, so that every MFMA sees other operand bits than the one before (the
// matrix cores draw more power, and the clock settles lower, on changing data than on a
// constant operand).
__global__ __launch_bounds__(256) void k_mfma_busy_loop(float *out, int iters) {
  bf16x8_t a[4], b[4];
  uint32_t x = 0x9e3779b9u * (threadIdx.x + 1);  // the same operands in every block
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      x ^= x << 13; x ^= x >> 17; x ^= x << 5;
      a[s][j] = (__bf16)((float)(x >> 8) * (2.0f / 16777216.0f) - 1.0f);
      x ^= x << 13; x ^= x >> 17; x ^= x << 5;
      b[s][j] = (__bf16)((float)(x >> 8) * (2.0f / 16777216.0f) - 1.0f);
    }
  f32x16_t acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  for (int it = 0; it < iters; it += 2) {
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i & 3], b[(i + 1) & 3], acc[i], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(i + 2) & 3], b[(i + 3) & 3], acc[i], 0, 0, 0);
  }
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) sum += acc[i][r];
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = sum;
}

hipError_t launch_mfma_busy_loop(int n_blocks, int iters, float *out, hipStream_t s) {
  if (n_blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_mfma_busy_loop, dim3(n_blocks), dim3(256), 0, s, out, iters);
  return hipGetLastError();
}

}  // namespace akvs
