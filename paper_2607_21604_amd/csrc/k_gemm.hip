// Projection GEMMs C = A . B^T (A [M][K] activations, B [N][K] weights) with fused
// epilogues: RoPE + q/k/v split (QKV), residual add into the fp32 stream (RESID),
// SiLU(gate) * up (SWIGLU) and plain stores.
//
// bf16 path: 128x128x64 block tiles, 4 waves in 2x2, each wave 64x64 from 2x2 MFMA
// 32x32x16 bf16 tiles with fp32 accumulation; operand tiles double-buffered in LDS,
// next tile prefetched into registers during the MFMA loop. The accumulator tile is
// staged through LDS so every epilogue can pair columns (rotary halves, gate/up) and
// write coalesced rows. fp32 path (small models): 32x128x32 VALU tiles, same epilogues.
#include <type_traits>

#include "kernels.h"

namespace akvs {

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// Epilogue over an LDS tile Cs[BM][ldc] holding C[m0.., n0..] (SWIGLU: gate cols [0,BN/2),
// up cols [BN/2,BN) of output columns n0..n0+BN/2).
template <int BM, int BN, int NT>
__device__ void epilogue_tile(const float *Cs, int ldc, int m0, int n0, int M_eff, int N,
                              const Epi &e) {
  const int tid = threadIdx.x;
  if (e.mode == EPI_STORE || e.mode == EPI_RESID) {
    constexpr int U = BN / 4;
    for (int idx = tid; idx < BM * U; idx += NT) {
      const int r = idx / U, c4 = (idx - (idx / U) * U) * 4;
      const int gm = m0 + r, gn = n0 + c4;
      if (gm >= M_eff || gn >= N) continue;
      const float *src = Cs + r * ldc + c4;
      if (e.mode == EPI_RESID) {
        float *hp = reinterpret_cast<float *>(e.out) + (size_t)gm * e.ldo + gn;
        float4 v = *reinterpret_cast<float4 *>(hp);
        v.x += src[0]; v.y += src[1]; v.z += src[2]; v.w += src[3];
        *reinterpret_cast<float4 *>(hp) = v;
      } else if (e.out_dtype == AKVS_BF16) {
        store4(reinterpret_cast<bf16_t *>(e.out) + (size_t)gm * e.ldo + gn, src[0], src[1], src[2], src[3]);
      } else {
        store4(reinterpret_cast<float *>(e.out) + (size_t)gm * e.ldo + gn, src[0], src[1], src[2], src[3]);
      }
    }
  } else if (e.mode == EPI_SWIGLU) {
    constexpr int HALF = BN / 2, U = HALF / 4;
    for (int idx = tid; idx < BM * U; idx += NT) {
      const int r = idx / U, c4 = (idx - (idx / U) * U) * 4;
      const int gm = m0 + r, gn = n0 + c4;
      if (gm >= M_eff || gn >= N) continue;
      const float *g = Cs + r * ldc + c4;
      const float *u = g + HALF;
      const float a0 = silu(g[0]) * u[0], a1 = silu(g[1]) * u[1];
      const float a2 = silu(g[2]) * u[2], a3 = silu(g[3]) * u[3];
      if (e.out_dtype == AKVS_BF16)
        store4(reinterpret_cast<bf16_t *>(e.out) + (size_t)gm * e.ldo + gn, a0, a1, a2, a3);
      else
        store4(reinterpret_cast<float *>(e.out) + (size_t)gm * e.ldo + gn, a0, a1, a2, a3);
    }
  } else {  // EPI_QKV: every tile holds whole heads of one section
    const int hd = e.hd, half = hd >> 1;
    const int lo_units = half >> 2;
    const int items = (BN / hd) * lo_units;  // per row
    const float2 *rope = reinterpret_cast<const float2 *>(e.rope);
    for (int idx = tid; idx < BM * items; idx += NT) {
      const int r = idx / items, it = idx - (idx / items) * items;
      const int hs = it / lo_units, u = it - hs * lo_units;
      const int gm = m0 + r;
      if (gm >= M_eff || n0 + hs * hd >= N) continue;
      const int col = e.n_off + n0 + hs * hd + u * 4;  // logical q|k|v column of the lo half
      const int pos = e.pos ? e.pos[gm] : e.pos0 + gm;
      const float *src = Cs + r * ldc + hs * hd + u * 4;
      float lo[4], hi[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        lo[i] = src[i];
        hi[i] = src[half + i];
      }
      if (col < e.hq_w + e.kv_w) {
        const int p = min(max(pos - e.rope_base, 0), e.rope_rows - 1);
        const float2 *rr = rope + (size_t)p * half + u * 4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float2 cs = rr[i];
          const float a = lo[i], b = hi[i];
          lo[i] = a * cs.x - b * cs.y;
          hi[i] = b * cs.x + a * cs.y;
        }
      }
      size_t off;
      void *base;
      if (col < e.hq_w) {
        base = e.q_out;
        off = (size_t)gm * e.hq_w + col;
      } else {
        const int drow = e.kv_by_pos ? pos : gm;
        if (col < e.hq_w + e.kv_w) {
          base = e.k_out;
          off = (size_t)drow * e.kv_w + (col - e.hq_w);
        } else {
          base = e.v_out;
          off = (size_t)drow * e.kv_w + (col - e.hq_w - e.kv_w);
        }
      }
      if (e.out_dtype == AKVS_BF16) {
        bf16_t *d = reinterpret_cast<bf16_t *>(base) + off;
        store4(d, lo[0], lo[1], lo[2], lo[3]);
        store4(d + half, hi[0], hi[1], hi[2], hi[3]);
      } else {
        float *d = reinterpret_cast<float *>(base) + off;
        store4(d, lo[0], lo[1], lo[2], lo[3]);
        store4(d + half, hi[0], hi[1], hi[2], hi[3]);
      }
    }
  }
}

// ------------------------------------------------------------------------------------------
// bf16 MFMA GEMM. Block tile BM x 128 x 64 (BM = 128 or 64), 256 threads as 2 x 2 waves, a
// wave owning (BM/2) x 64 outputs as (BM/64) x 2 tiles of v_mfma_f32_32x32x16_bf16.
// Operand tiles: two LDS buffers (rows padded to 144 B: the 16 rows one ds_read_b128 phase
// touches fall on distinct banks) and two register stages, so the global loads of tile
// kt+2 are in flight while tile kt is multiplied and tile kt+1 is written to LDS.
constexpr int GB_N = 128, GB_K = 64;

template <bool MF16>
__device__ __forceinline__ typename std::conditional<MF16, f32x4_t, f32x16_t>::type mfma_tile(
    bf16x8_t a, bf16x8_t b, typename std::conditional<MF16, f32x4_t, f32x16_t>::type c);
template <>
__device__ __forceinline__ f32x4_t mfma_tile<true>(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
template <>
__device__ __forceinline__ f32x16_t mfma_tile<false>(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
constexpr int G_LDS = GB_K + 8;  // bf16 per LDS row
constexpr int G_NS = 3;          // register prefetch stages
constexpr int G_CLD = GB_N + 4;  // fp32 C tile row stride

// K splits for a grid of `tiles` output tiles, n_slots = 2 x compute units (two resident
// blocks each): grids that would leave at least half of the units idle are split so that
// every unit gets about two items, each split keeping >= 4 k-steps of 64.
__host__ __device__ inline int gemm_k_splits(int tiles, int nk, int n_slots) {
  // measured: only long reductions (K >= 6144) gain from the extra partial-tile traffic,
  // and only on small grids: a grid of about one tile per unit (the 3B down-projection of
  // ~1400 rows, 264 tiles) ran 12 % faster unsplit than split in two plus the fixup pass
  if (tiles <= 0 || nk < 96 || 4 * tiles > n_slots) return 1;
  int sp = (n_slots + tiles - 1) / tiles;
  const int cap = nk / 4;
  if (sp > cap) sp = cap;
  if (sp > 64) sp = 64;
  return sp < 2 ? 1 : sp;
}

template <int BM, bool MF16>
struct GemmShape {
  static constexpr int A_CH = BM * GB_K / 8 / 256;     // 16-byte A chunks per thread
  static constexpr int B_CH = GB_N * GB_K / 8 / 256;   // 16-byte B chunks per thread
  static constexpr int A_TILE = BM * G_LDS;            // bf16 elements
  static constexpr int B_TILE = GB_N * G_LDS;
  static constexpr int BUF = A_TILE + B_TILE;
  static constexpr int LOOP_BYTES = 2 * BUF * 2;
  static constexpr int C_BYTES = BM * G_CLD * 4;
  static constexpr int SMEM = LOOP_BYTES > C_BYTES ? LOOP_BYTES : C_BYTES;
  // per wave (BM/2) x 64 outputs: MF16 -> (BM/32) x 4 tiles of 16x16, else (BM/64) x 2 of 32x32
  static constexpr int MT = MF16 ? 16 : 32;
  static constexpr int MI = (BM / 2) / MT;
  static constexpr int NJ = 64 / MT;
  static constexpr int KSTEP = MF16 ? 32 : 16;
};

// Blocks form a 1-D grid over (tile, k-split) work items decoded on the device from the
// live row count. With k_splits > 1 every tile's K range is cut in k_splits slices whose
// fp32 partial tiles go to `part` ([tile][split][BM][128]); k_gemm_fixup then adds them in
// split order and runs the epilogue. k_splits follows gemm_k_splits(live tile count).
template <int BM, bool MF16>
__global__ __launch_bounds__(256, 2) void k_gemm_bf16(const bf16_t *__restrict__ A, int lda,
                                                      const bf16_t *__restrict__ B, int ldb,
                                                      int M, int N, int K,
                                                      const int32_t *m_dev, Epi epi,
                                                      int n_slots, float *__restrict__ part) {
  using S = GemmShape<BM, MF16>;
  using AccT = typename std::conditional<MF16, f32x4_t, f32x16_t>::type;
  constexpr int ACC_N = MF16 ? 4 : 16;
  __shared__ __attribute__((aligned(16))) unsigned char smem[S::SMEM];
  bf16_t *sm = reinterpret_cast<bf16_t *>(smem);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int M_eff = M;
  if (m_dev) M_eff = min(M, *m_dev);
  const bool swiglu = epi.mode == EPI_SWIGLU;
  const int bn_out = swiglu ? GB_N / 2 : GB_N;
  const int n_tiles = (N + bn_out - 1) / bn_out;
  const int tiles = ((M_eff + BM - 1) / BM) * n_tiles;
  const int nk = K / GB_K;
  const int splits = part ? gemm_k_splits(tiles, nk, n_slots) : 1;
  const int item = blockIdx.x;
  if (item >= tiles * splits) return;
  const int tile = item / splits, split = item - tile * splits;
  const int m0 = (tile / n_tiles) * BM;
  const int n0 = (tile - (tile / n_tiles) * n_tiles) * bn_out;
  const int k_per = (nk + splits - 1) / splits;
  const int kt0 = min(nk, split * k_per), kt1 = min(nk, kt0 + k_per);
  const int nkt = kt1 - kt0;

  // Per-thread 16-byte chunks: chunk c = tid + 256 i covers row c / 8, k columns
  // (c % 8) * 8 ..+7. Rows past M / N are clamped to a valid row: they only feed
  // accumulator rows / columns the epilogue discards.
  size_t a_off[S::A_CH], b_off[S::B_CH];
  int la_off[S::A_CH], lb_off[S::B_CH];
#pragma unroll
  for (int i = 0; i < S::A_CH; ++i) {
    const int c = tid + 256 * i;
    const int r = c >> 3, kc = (c & 7) * 8;
    a_off[i] = (size_t)min(m0 + r, M_eff - 1) * lda + kc;
    la_off[i] = r * G_LDS + kc;
  }
#pragma unroll
  for (int i = 0; i < S::B_CH; ++i) {
    const int c = tid + 256 * i;
    const int r = c >> 3, kc = (c & 7) * 8;
    int gn;
    if (swiglu) {
      const int oc = min(n0 + (r & 63), N - 1);
      gn = (r < 64) ? oc : N + oc;
    } else {
      gn = min(n0 + r, N - 1);
    }
    b_off[i] = (size_t)gn * ldb + kc;
    lb_off[i] = S::A_TILE + r * G_LDS + kc;
  }

  AccT acc[S::MI][S::NJ];
#pragma unroll
  for (int i = 0; i < S::MI; ++i)
#pragma unroll
    for (int j = 0; j < S::NJ; ++j)
#pragma unroll
      for (int r = 0; r < ACC_N; ++r) acc[i][j][r] = 0.f;

  // three register stages (ring slots) of operand chunks in flight
  u32x4_t ra[G_NS][S::A_CH], rb[G_NS][S::B_CH];

#define AKVS_GLOAD(SL, KT)                                                          \
  {                                                                                 \
    const int k0_ = (KT) * GB_K;                                                    \
    _Pragma("unroll") for (int i = 0; i < S::A_CH; ++i)                             \
        ra[SL][i] = *reinterpret_cast<const u32x4_t *>(A + a_off[i] + k0_);         \
    _Pragma("unroll") for (int i = 0; i < S::B_CH; ++i)                             \
        rb[SL][i] = *reinterpret_cast<const u32x4_t *>(B + b_off[i] + k0_);         \
  }
#define AKVS_SSTORE(SL, BUFI)                                                       \
  {                                                                                 \
    bf16_t *base_ = sm + (BUFI) * S::BUF;                                           \
    _Pragma("unroll") for (int i = 0; i < S::A_CH; ++i)                             \
        *reinterpret_cast<u32x4_t *>(base_ + la_off[i]) = ra[SL][i];                \
    _Pragma("unroll") for (int i = 0; i < S::B_CH; ++i)                             \
        *reinterpret_cast<u32x4_t *>(base_ + lb_off[i]) = rb[SL][i];                \
  }
#define AKVS_COMPUTE(BUFI)                                                                    \
  {                                                                                           \
    const bf16_t *As_ = sm + (BUFI) * S::BUF;                                                 \
    const bf16_t *Bs_ = As_ + S::A_TILE;                                                      \
    _Pragma("unroll") for (int ks = 0; ks < GB_K / S::KSTEP; ++ks) {                          \
      bf16x8_t af[S::MI], bfr[S::NJ];                                                         \
      const int kk = ks * S::KSTEP + (lane / S::MT) * 8;                                      \
      _Pragma("unroll") for (int i = 0; i < S::MI; ++i) af[i] =                               \
          *reinterpret_cast<const bf16x8_t *>(                                                \
              As_ + (wm * (BM / 2) + i * S::MT + (lane % S::MT)) * G_LDS + kk);                \
      _Pragma("unroll") for (int j = 0; j < S::NJ; ++j) bfr[j] =                              \
          *reinterpret_cast<const bf16x8_t *>(Bs_ + (wn * 64 + j * S::MT + (lane % S::MT)) *  \
                                                        G_LDS + kk);                          \
      _Pragma("unroll") for (int i = 0; i < S::MI; ++i)                                       \
          _Pragma("unroll") for (int j = 0; j < S::NJ; ++j) acc[i][j] = mfma_tile<MF16>(      \
              af[i], bfr[j], acc[i][j]);                                                      \
    }                                                                                         \
  }

  // One k-step: multiply the tile in LDS buffer u&1, move the next tile from its ring
  // slot to the other buffer, then refill that slot G_NS tiles ahead. Loads past the
  // range re-read its last tile, so every load is unconditional and the compiler's
  // count of outstanding loads stays exact (each wait only covers the oldest stage);
  // the scheduling barrier keeps the refill ahead of the next step's LDS traffic.
#define AKVS_STEP(U, J)                                                             \
  {                                                                                 \
    AKVS_COMPUTE((U) & 1);                                                          \
    AKVS_SSTORE(((U) + 1) % G_NS, ((U) + 1) & 1);                                   \
    __syncthreads();                                                                \
    AKVS_GLOAD(((U) + 1) % G_NS, min(kt0 + (J) + 1 + G_NS, kl));                    \
    __builtin_amdgcn_sched_barrier(0);                                              \
  }
  const int kl = kt1 - 1;  // kt1 >= 1: a valid tile even for an empty range
#pragma unroll
  for (int sl = 0; sl < G_NS; ++sl) AKVS_GLOAD(sl, min(kt0 + sl, kl));
  AKVS_SSTORE(0, 0);
  AKVS_GLOAD(0, min(kt0 + G_NS, kl));
  __syncthreads();
  constexpr int UNR = 2 * G_NS;  // ring slot and LDS buffer both return to 0
  int j = 0;
  for (; j + UNR <= nkt; j += UNR) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) AKVS_STEP(u, j + u);
  }
#pragma unroll
  for (int u = 0; u < UNR; ++u)
    if (j + u < nkt) AKVS_STEP(u, j + u);
#undef AKVS_STEP
#undef AKVS_GLOAD
#undef AKVS_SSTORE
#undef AKVS_COMPUTE

  // split K: the partial tile goes to the workspace, k_gemm_fixup finishes it
  float *Cs = splits > 1 ? part + (size_t)item * BM * GB_N : reinterpret_cast<float *>(smem);
  const int ldc = splits > 1 ? GB_N : G_CLD;
#pragma unroll
  for (int i = 0; i < S::MI; ++i)
#pragma unroll
    for (int j = 0; j < S::NJ; ++j)
#pragma unroll
      for (int r = 0; r < ACC_N; ++r) {
        // 32x32 tile: row (r/4)*8 + (lane/32)*4 + r%4; 16x16 tile: row (lane/16)*4 + r
        const int trow = MF16 ? (lane >> 4) * 4 + r : (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        const int row = wm * (BM / 2) + i * S::MT + trow;
        const int col = wn * 64 + j * S::MT + (lane % S::MT);
        Cs[row * ldc + col] = acc[i][j][r];
      }
  if (splits > 1) return;
  __syncthreads();
  epilogue_tile<BM, GB_N, 256>(Cs, G_CLD, m0, n0, M_eff, N, epi);
}

// Second pass of a K-split GEMM: a block takes G_FR rows of one tile, adds their partial
// rows in split order into an LDS slice and runs the epilogue on it.
constexpr int G_FR = 16;
template <int BM>
__global__ __launch_bounds__(256) void k_gemm_fixup(int M, int N, int K, const int32_t *m_dev,
                                                    Epi epi, int n_slots,
                                                    const float *__restrict__ part) {
  __shared__ __attribute__((aligned(16))) float Cs[G_FR * G_CLD];
  int M_eff = M;
  if (m_dev) M_eff = min(M, *m_dev);
  const bool swiglu = epi.mode == EPI_SWIGLU;
  const int bn_out = swiglu ? GB_N / 2 : GB_N;
  const int n_tiles = (N + bn_out - 1) / bn_out;
  const int tiles = ((M_eff + BM - 1) / BM) * n_tiles;
  const int splits = gemm_k_splits(tiles, K / GB_K, n_slots);
  constexpr int SLICES = BM / G_FR;
  const int tile = blockIdx.x / SLICES, slice = blockIdx.x - tile * SLICES;
  if (splits < 2 || tile >= tiles) return;
  const int m0 = (tile / n_tiles) * BM + slice * G_FR;
  if (m0 >= M_eff) return;
  const int n0 = (tile - (tile / n_tiles) * n_tiles) * bn_out;
  const float *src = part + (size_t)tile * splits * BM * GB_N + (size_t)slice * G_FR * GB_N;
  constexpr int PER = G_FR * GB_N / 4 / 256;  // float4 per thread
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e4 = threadIdx.x + 256 * i;
    const int row = e4 / (GB_N / 4), c4 = (e4 - row * (GB_N / 4)) * 4;
    const float *p = src + row * GB_N + c4;
    float4 acc = *reinterpret_cast<const float4 *>(p);
    for (int sp = 1; sp < splits; ++sp) {
      const float4 v = *reinterpret_cast<const float4 *>(p + (size_t)sp * BM * GB_N);
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
    *reinterpret_cast<float4 *>(Cs + row * G_CLD + c4) = acc;
  }
  __syncthreads();
  epilogue_tile<G_FR, GB_N, 256>(Cs, G_CLD, m0, n0, M_eff, N, epi);
}

// ------------------------------------------------------------------------------------------
// fp32 VALU GEMM (small fp32 models). 32x128 tile, BK 32, thread = 4 rows x 4 columns.
constexpr int GF_M = 32, GF_N = 128, GF_K = 32;

__global__ __launch_bounds__(256) void k_gemm_f32(const float *__restrict__ A, int lda,
                                                  const float *__restrict__ B, int ldb, int M,
                                                  int N, int K, const int32_t *m_dev, Epi epi) {
  __shared__ __attribute__((aligned(16))) float smem[GF_M * (GF_N + 4) > GF_K * (GF_M + GF_N + 8)
                                                        ? GF_M * (GF_N + 4)
                                                        : GF_K * (GF_M + GF_N + 8)];
  float *As = smem;                    // [GF_K][GF_M + 4]  (k-major)
  float *Bs = smem + GF_K * (GF_M + 4);  // [GF_K][GF_N + 4]
  const int tid = threadIdx.x;
  int M_eff = M;
  if (m_dev) M_eff = min(M, *m_dev);
  const int m0 = blockIdx.y * GF_M;
  if (m0 >= M_eff) return;
  const bool swiglu = epi.mode == EPI_SWIGLU;
  const int n0 = blockIdx.x * (swiglu ? GF_N / 2 : GF_N);
  const int tr = tid >> 5, tc = tid & 31;  // rows tr*4.., cols tc*4..
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += GF_K) {
    __syncthreads();
    {  // A: 32 rows x 32 k = 256 float4, one per thread
      const int r = tid >> 3, kc = (tid & 7) * 4;
      const int gm = m0 + r, gk = k0 + kc;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (gm < M_eff && gk < K) v = *reinterpret_cast<const float4 *>(A + (size_t)gm * lda + gk);
      As[(kc + 0) * (GF_M + 4) + r] = v.x;
      As[(kc + 1) * (GF_M + 4) + r] = v.y;
      As[(kc + 2) * (GF_M + 4) + r] = v.z;
      As[(kc + 3) * (GF_M + 4) + r] = v.w;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {  // B: 128 rows x 32 k = 1024 float4
      const int c = tid + 256 * i;
      const int r = c >> 3, kc = (c & 7) * 4;
      int gn;
      bool ok;
      if (swiglu) {
        const int oc = n0 + (r & 63);
        ok = oc < N;
        gn = (r < 64) ? oc : N + oc;
      } else {
        gn = n0 + r;
        ok = gn < N;
      }
      const int gk = k0 + kc;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (ok && gk < K) v = *reinterpret_cast<const float4 *>(B + (size_t)gn * ldb + gk);
      Bs[(kc + 0) * (GF_N + 4) + r] = v.x;
      Bs[(kc + 1) * (GF_N + 4) + r] = v.y;
      Bs[(kc + 2) * (GF_N + 4) + r] = v.z;
      Bs[(kc + 3) * (GF_N + 4) + r] = v.w;
    }
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < GF_K; ++k) {
      const float4 a = *reinterpret_cast<const float4 *>(As + k * (GF_M + 4) + tr * 4);
      const float4 b = *reinterpret_cast<const float4 *>(Bs + k * (GF_N + 4) + tc * 4);
      const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
  }
  __syncthreads();
  float *Cs = smem;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) Cs[(tr * 4 + i) * (GF_N + 4) + tc * 4 + j] = acc[i][j];
  __syncthreads();
  epilogue_tile<GF_M, GF_N, 256>(Cs, GF_N + 4, m0, n0, M_eff, N, epi);
}

int gemm_cu_count() {
  static int n = 0;
  if (n == 0) {
    int dev = 0, cu = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cu > 0)
      n = cu;
    else
      n = 256;
  }
  return n;
}

size_t gemm_part_floats(int M, int N, int K, int mode) {
  const int bn = mode == EPI_SWIGLU ? GB_N / 2 : GB_N;
  const int tiles_cap = ((N + bn - 1) / bn) * ((M + 127) / 128);
  const int n_slots = 2 * gemm_cu_count();
  size_t items = 0;
  for (int t = 1; t <= tiles_cap; ++t) {
    const int sp = gemm_k_splits(t, K / GB_K, n_slots);
    if (sp > 1 && (size_t)t * sp > items) items = (size_t)t * sp;
  }
  return items * 128 * GB_N;
}

// Grid of the bf16 GEMM: work items (tile x K-split) for every row count the host cannot
// rule out (exactly M without a device count, else [m_min, M]); n_slots = 0 when no such
// count splits K, so the device never splits either.
struct GemmPlan {
  int items, tiles_cap, n_slots;
  bool any_split;
};
static GemmPlan gemm_plan(int M, int N, int K, const int32_t *m_dev, const Epi &epi,
                          const float *part, int m_min) {
  const int bn = epi.mode == EPI_SWIGLU ? GB_N / 2 : GB_N;
  const int n_tiles = (N + bn - 1) / bn;
  GemmPlan p;
  p.tiles_cap = n_tiles * ((M + 127) / 128);
  p.items = p.tiles_cap;
  p.any_split = false;
  p.n_slots = part ? 2 * gemm_cu_count() : 0;
  if (part) {
    const int lo = m_dev ? (m_min > 1 ? m_min : 1) : M;
    for (int t = n_tiles * ((lo + 127) / 128); t <= p.tiles_cap; ++t) {
      const int sp = gemm_k_splits(t, K / GB_K, p.n_slots);
      p.any_split |= sp > 1;
      if (t * sp > p.items) p.items = t * sp;
    }
    if (!p.any_split) p.n_slots = 0;
  }
  return p;
}

hipError_t launch_gemm(const void *A, int lda, const void *B, int ldb, int M, int N, int K,
                       const int32_t *m_dev, int dtype, const Epi &epi, hipStream_t s,
                       float *part, int m_min) {
  if (M == 0 || N == 0) return hipSuccess;
  if (dtype == AKVS_BF16) {
    const GemmPlan p = gemm_plan(M, N, K, m_dev, epi, part, m_min);
    hipLaunchKernelGGL((k_gemm_bf16<128, false>), dim3(p.items), dim3(256), 0, s,
                       reinterpret_cast<const bf16_t *>(A), lda,
                       reinterpret_cast<const bf16_t *>(B), ldb, M, N, K, m_dev, epi, p.n_slots,
                       part);
  } else {
    const bool swiglu = epi.mode == EPI_SWIGLU;
    const int bn = swiglu ? GF_N / 2 : GF_N;
    dim3 g((N + bn - 1) / bn, (M + GF_M - 1) / GF_M), b(256);
    hipLaunchKernelGGL(k_gemm_f32, g, b, 0, s, reinterpret_cast<const float *>(A), lda,
                       reinterpret_cast<const float *>(B), ldb, M, N, K, m_dev, epi);
  }
  return hipGetLastError();
}

hipError_t launch_gemm_fixup(const void *, int, const void *, int, int M, int N, int K,
                             const int32_t *m_dev, int dtype, const Epi &epi, hipStream_t s,
                             float *part, int m_min) {
  if (M == 0 || N == 0 || dtype != AKVS_BF16) return hipSuccess;
  const GemmPlan p = gemm_plan(M, N, K, m_dev, epi, part, m_min);
  if (!p.any_split) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_fixup<128>), dim3(p.tiles_cap * (128 / G_FR)), dim3(256), 0, s, M,
                     N, K, m_dev, epi, p.n_slots, part);
  return hipGetLastError();
}

}  // namespace akvs
