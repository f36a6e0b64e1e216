// Attention of (sparse, position-sorted) query rows over a causal key range.
//
// bf16 path: one block = the query heads of one KV head over a tile of rows; each wave owns
// 16 rows of one query head. Keys stream through LDS in tiles of 64 (K row-major, V
// transposed), shared by every wave of the block. Scores are computed transposed,
// S^T = K Q^T, with MFMA 16x16x32 bf16: each lane then holds 16 scores of ONE query row,
// so the online softmax needs only two cross-lane steps, and the probabilities already
// sit in the operand layout of the second product O^T = V^T P^T (the pairing of the
// 32 contraction slots with keys is a fixed permutation applied to both operands).
// Row tiles are launched longest-first (rows are sorted by position, so later tiles
// see more keys).
#include "kernels.h"

namespace akvs {

// A block serves one KV head: RB query rows x all G query heads that read it. Wave w owns
// 16 rows (row block w / G) of query head w % G; NW = (RB / 16) * G waves (<= 12). Waves 0-3
// stage each 64-key K / V tile in LDS for all of them (double buffered, next tile
// prefetched into registers during the current one). Block b serves KV head b % Hkv, so
// the blocks streaming one head's keys run on the same XCD and share its L2.
// Column (bf16 element) of key group g (4 keys) in row r of the V^T tile (rows of 64
// elements, no padding). The XOR swizzle makes every 16-lane pass of both the transposed
// 8-byte writes and the 8-byte fragment reads touch 32 distinct 4-byte banks.
__device__ __forceinline__ int vt_col(int r, int g) { return (g ^ ((r ^ (r >> 3)) & 15)) * 4; }

template <int HD>
__global__ __launch_bounds__(768) void k_attn_bf16(const bf16_t *__restrict__ Q,
                                                   const int32_t *pos, int pos0, int rows,
                                                   const int32_t *rows_dev,
                                                   const bf16_t *__restrict__ Kc,
                                                   const bf16_t *__restrict__ Vc, int n_keys,
                                                   int hq, int hkv, int rb_rows, int n_tiles,
                                                   int n_splits, int split_keys,
                                                   float scale_log2, bf16_t *__restrict__ out,
                                                   float *__restrict__ part_o,
                                                   float *__restrict__ part_ml) {
  constexpr int KS = HD / 32;          // contraction steps of S
  constexpr int HB = HD / 16;          // 16-wide head-dim blocks of O
  constexpr int KST = HD + 8;          // K tile row stride (bf16)
  constexpr int VST = 64;              // V^T tile row stride (bf16), swizzled by vt_col
  constexpr int CPK = HD / 8;          // 16-byte chunks per key row
  constexpr int KCH = 64 * CPK / 256;  // K chunks per loading thread
  constexpr int VKEYS = CPK / 4;       // keys per loading thread in the V transpose
  constexpr int KBUF = 64 * KST, VBUF = HD * VST;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2 * KBUF];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[2 * VBUF];
  __shared__ int s_max[12];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nw = blockDim.x >> 6;
  const bool loader = wave < 4;
  const int G = hq / hkv;
  const int kvh = blockIdx.x % hkv;
  const int rest = (int)(blockIdx.x / hkv);
  const int split = rest % n_splits;
  const int tile = n_tiles - 1 - rest / n_splits;
  const int head = kvh * G + wave % G;
  int R = rows;
  if (rows_dev) R = min(R, *rows_dev);
  const int row0 = tile * rb_rows;
  if (tile < 0 || row0 >= R) return;
  const int r = row0 + (wave / G) * 16 + (lane & 15);
  const bool rvalid = r < R;
  const int rp = rvalid ? (pos ? pos[r] : pos0 + r) : -1;
  const int rpos = rvalid ? rp : 0;
  int wmax = rp;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) wmax = max(wmax, __shfl_xor(wmax, o, 64));
  if (lane == 0) s_max[wave] = wmax;
  __syncthreads();
  int bmax = -1;
  for (int w = 0; w < nw; ++w) bmax = max(bmax, s_max[w]);
  // this block's keys: [kv_begin, kv_end) of split `split`
  const int kv_begin = split * split_keys;
  const int kv_end = min(min(n_keys, bmax + 1), kv_begin + split_keys);
  const int nkt = kv_end > kv_begin ? (kv_end - kv_begin + 63) / 64 : 0;
  const size_t prow = ((size_t)split * rows + r) * hq + head;  // partial slot of this lane's row
  if (nkt == 0) {
    if (n_splits > 1 && rvalid && lane < 16) {
      part_ml[2 * prow] = -INFINITY;
      part_ml[2 * prow + 1] = 0.f;
    }
    return;
  }

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

  // One K / V tile in the loading waves' registers. Keys past kv_end are clamped to the
  // last key: finite data that the score mask gives probability 0.
  u32x4_t kreg[KCH], vreg[VKEYS];
  const int vkg = tid / CPK, ve0 = (tid - vkg * CPK) * 8;  // V: keys vkg*VKEYS.., dims ve0..
  const int klast = kv_end - 1;
#define AKVS_KV_LOAD(KEY0)                                                                  \
  {                                                                                         \
    _Pragma("unroll") for (int i = 0; i < KCH; ++i) {                                       \
      const int c = tid + 256 * i, kr = c / CPK, e0 = (c - kr * CPK) * 8;                   \
      const int key = min((KEY0) + kr, klast);                                              \
      kreg[i] = *reinterpret_cast<const u32x4_t *>(Kc + ((size_t)key * hkv + kvh) * HD + e0); \
    }                                                                                       \
    _Pragma("unroll") for (int j = 0; j < VKEYS; ++j) {                                     \
      const int key = min((KEY0) + vkg * VKEYS + j, klast);                                 \
      vreg[j] = *reinterpret_cast<const u32x4_t *>(Vc + ((size_t)key * hkv + kvh) * HD + ve0); \
    }                                                                                       \
  }
#define AKVS_KV_STORE(BUFI)                                                                 \
  {                                                                                         \
    bf16_t *ks_ = Ks + (BUFI) * KBUF;                                                       \
    bf16_t *vt_ = Vt + (BUFI) * VBUF;                                                       \
    _Pragma("unroll") for (int i = 0; i < KCH; ++i) {                                       \
      const int c = tid + 256 * i, kr = c / CPK, e0 = (c - kr * CPK) * 8;                   \
      *reinterpret_cast<u32x4_t *>(ks_ + kr * KST + e0) = kreg[i];                          \
    }                                                                                       \
    _Pragma("unroll") for (int d = 0; d < 8; ++d) {                                         \
      const int word = d >> 1;                                                              \
      const bool hi_ = (d & 1) != 0;                                                        \
      if (VKEYS == 4) {                                                                     \
        const uint32_t a0 = vreg[0][word], a1 = vreg[1][word];                              \
        const uint32_t a2 = vreg[VKEYS > 2 ? 2 : 0][word], a3 = vreg[VKEYS > 3 ? 3 : 0][word]; \
        uint2 v2;                                                                           \
        v2.x = hi_ ? ((a0 >> 16) | (a1 & 0xffff0000u)) : ((a0 & 0xffffu) | (a1 << 16));    \
        v2.y = hi_ ? ((a2 >> 16) | (a3 & 0xffff0000u)) : ((a2 & 0xffffu) | (a3 << 16));    \
        *reinterpret_cast<uint2 *>(vt_ + (ve0 + d) * VST + vt_col(ve0 + d, vkg)) = v2;     \
      } else {                                                                              \
        const uint32_t a0 = vreg[0][word], a1 = vreg[VKEYS > 1 ? 1 : 0][word];              \
        *reinterpret_cast<uint32_t *>(vt_ + (ve0 + d) * VST + vt_col(ve0 + d, vkg >> 1) +     \
                                      (vkg & 1) * 2) =                                      \
            hi_ ? ((a0 >> 16) | (a1 & 0xffff0000u)) : ((a0 & 0xffffu) | (a1 << 16));        \
      }                                                                                     \
    }                                                                                       \
  }

  if (loader) {
    AKVS_KV_LOAD(kv_begin);
    AKVS_KV_STORE(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int key0 = kv_begin + kt * 64;
    const bool more = kt + 1 < nkt;
    if (loader && more) AKVS_KV_LOAD(key0 + 64);
    const bf16_t *ks_ = Ks + (kt & 1) * KBUF;
    const bf16_t *vt_ = Vt + (kt & 1) * VBUF;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int sk0 = key0 + st * 32;
      if (sk0 <= wmax) {  // skip keys past every row of this wave
        f32x4_t s[2];
        s[0] = s[1] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2) {
          const bf16_t *krow = ks_ + ((st * 2 + kb2) * 16 + (lane & 15)) * KST + (lane >> 4) * 8;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const bf16x8_t a = *reinterpret_cast<const bf16x8_t *>(krow + ks * 32);
            s[kb2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[ks], s[kb2], 0, 0, 0);
          }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = sk0 + kb2 * 16 + (lane >> 4) * 4 + i;
            const float v = (key > rpos || key >= kv_end) ? -INFINITY : s[kb2][i] * scale_log2;
            s[kb2][i] = v;
            mx = fmaxf(mx, v);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run, mx);
        // rows with no key yet in this split keep m = -inf; offset by 0 then (p, alpha = 0)
        const float m_off = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(m_run - m_off);
        float rs = 0.f;
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float p = exp2f(s[kb2][i] - m_off);
            s[kb2][i] = p;
            rs += p;
          }
        rs += __shfl_xor(rs, 16, 64);
        rs += __shfl_xor(rs, 32, 64);
        l_run = l_run * alpha + rs;
        m_run = m_new;
#pragma unroll
        for (int hb = 0; hb < HB; ++hb) o[hb] *= alpha;
        uint32_t pw[4];
        pw[0] = pack_bf2(s[0][0], s[0][1]);
        pw[1] = pack_bf2(s[0][2], s[0][3]);
        pw[2] = pack_bf2(s[1][0], s[1][1]);
        pw[3] = pack_bf2(s[1][2], s[1][3]);
        bf16x8_t pb;
        __builtin_memcpy(&pb, pw, 16);
#pragma unroll
        for (int hb = 0; hb < HB; ++hb) {
          const int vr = hb * 16 + (lane & 15);
          const bf16_t *vrow = vt_ + vr * VST;
          const int kg = st * 8 + (lane >> 4);
          uint32_t vw[4];
          const uint2 x0 = *reinterpret_cast<const uint2 *>(vrow + vt_col(vr, kg));
          const uint2 x1 = *reinterpret_cast<const uint2 *>(vrow + vt_col(vr, kg + 4));
          vw[0] = x0.x; vw[1] = x0.y; vw[2] = x1.x; vw[3] = x1.y;
          bf16x8_t a;
          __builtin_memcpy(&a, vw, 16);
          o[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb, o[hb], 0, 0, 0);
        }
      }
    }
    if (loader && more) AKVS_KV_STORE((kt + 1) & 1);
    __syncthreads();
  }
#undef AKVS_KV_LOAD
#undef AKVS_KV_STORE
  if (!rvalid) return;
  if (n_splits > 1) {  // unnormalised partial + (max, sum) for the combine pass
    float *po = part_o + prow * HD + (lane >> 4) * 4;
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) store4(po + hb * 16, o[hb][0], o[hb][1], o[hb][2], o[hb][3]);
    if (lane < 16) {
      part_ml[2 * prow] = m_run;
      part_ml[2 * prow + 1] = l_run;
    }
    return;
  }
  const float inv = 1.0f / l_run;
  bf16_t *orow = out + ((size_t)r * hq + head) * HD + (lane >> 4) * 4;
#pragma unroll
  for (int hb = 0; hb < HB; ++hb)
    store4(orow + hb * 16, o[hb][0] * inv, o[hb][1] * inv, o[hb][2] * inv, o[hb][3] * inv);
}

// Merge of the key splits of one (row, head): weights 2^(m_s - max m), fixed split order.
__global__ __launch_bounds__(256) void k_attn_combine(const float *__restrict__ part_o,
                                                      const float *__restrict__ part_ml,
                                                      int n_splits, int rows,
                                                      const int32_t *rows_dev, int hq, int hd,
                                                      bf16_t *__restrict__ out) {
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);  // (row, head), one wave each
  const int lane = threadIdx.x & 63;
  int R = rows;
  if (rows_dev) R = min(R, *rows_dev);
  if (item >= R * hq) return;
  float mx = -INFINITY;
  for (int sp = 0; sp < n_splits; ++sp) mx = fmaxf(mx, part_ml[2 * ((size_t)sp * rows * hq + item)]);
  const float moff = mx == -INFINITY ? 0.f : mx;
  float l = 0.f, a0 = 0.f, a1 = 0.f;
  for (int sp = 0; sp < n_splits; ++sp) {
    const size_t pi = (size_t)sp * rows * hq + item;
    const float w = exp2f(part_ml[2 * pi] - moff);
    l += w * part_ml[2 * pi + 1];
    const float *po = part_o + pi * hd;
    a0 += w * po[lane];
    if (hd > 64) a1 += w * po[lane + 64];
  }
  const float inv = 1.0f / l;
  out[(size_t)item * hd + lane] = f2bf(a0 * inv);
  if (hd > 64) out[(size_t)item * hd + lane + 64] = f2bf(a1 * inv);
}

// Rows per block of the bf16 kernel for G query heads per KV head (0: not supported).
static inline int attn_block_rows(int G) {
  if (G < 1 || G > 12) return 0;
  const int rb = 12 / G;
  return 16 * (rb > 4 ? 4 : rb);
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

int attn_splits(int rows, int hq, int hkv, int n_keys) {
  const int rb = attn_block_rows(hq / hkv);
  if (rb == 0 || rows <= 0) return 1;
  const long long base = (long long)((rows + rb - 1) / rb) * hkv;
  long long sp = (512 + base - 1) / base;           // aim at ~512 blocks
  const long long cap = (n_keys + 255) / 256;        // at least 256 keys per split
  if (sp > cap) sp = cap;
  if (sp > 64) sp = 64;
  return sp < 1 ? 1 : (int)sp;
}

int attn_split_keys(int n_keys, int n_splits) {
  const int per = (n_keys + n_splits - 1) / n_splits;
  return (per + 63) / 64 * 64;
}

hipError_t launch_attention(const void *q, const int32_t *pos, int pos0, int rows,
                            const int32_t *rows_dev, const void *k, const void *v, int n_keys,
                            int hq, int hkv, int hd, int dtype, void *out, float *part_o,
                            float *part_ml, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (dtype == AKVS_BF16) {
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    const bf16_t *Q = reinterpret_cast<const bf16_t *>(q);
    const bf16_t *K = reinterpret_cast<const bf16_t *>(k);
    const bf16_t *V = reinterpret_cast<const bf16_t *>(v);
    bf16_t *O = reinterpret_cast<bf16_t *>(out);
    const int G = hq / hkv;
    const int rb = attn_block_rows(G);
    if (rb == 0) return hipErrorInvalidValue;
    const int n_tiles = (rows + rb - 1) / rb;
    const int n_splits = part_o ? attn_splits(rows, hq, hkv, n_keys) : 1;
    const int split_keys = attn_split_keys(n_keys, n_splits);
    dim3 g(n_tiles * hkv * n_splits), b(64 * (rb / 16) * G);
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_bf16<128>, g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V, n_keys,
                         hq, hkv, rb, n_tiles, n_splits, split_keys, scale_log2, O, part_o,
                         part_ml);
    else
      hipLaunchKernelGGL(k_attn_bf16<64>, g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V, n_keys,
                         hq, hkv, rb, n_tiles, n_splits, split_keys, scale_log2, O, part_o,
                         part_ml);
    if (n_splits > 1) {
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      const long long items = (long long)rows * hq;
      hipLaunchKernelGGL(k_attn_combine, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, s,
                         part_o, part_ml, n_splits, rows, rows_dev, hq, hd, O);
    }
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
