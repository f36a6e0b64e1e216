// Projection GEMMs C = A . B^T (A [M][K] activations, B [N][K] weights) with fused
// epilogues: RoPE + q/k/v split (QKV), residual add into the fp32 stream (RESID),
// SiLU(gate) * up (SWIGLU) and plain stores.
//
// bf16 path, three kernels on v_mfma_f32_32x32x16_bf16 with fp32 accumulation, operand
// tiles double-buffered in LDS and fed by register stages of global loads:
//   k_gemm_bf16_w8 - 8 waves, BM x BN x 64 tiles (256/192 x 256/128), all waves on one
//                    schedule interleaving loads, LDS stores and MFMAs;
//   k_gemm_bf16_pp - 8 waves, 192 x 256 tiles, two wave groups alternating memory and
//                    MFMA phases ("ping-pong");
//   k_gemm_bf16    - 4 waves, 128 x 128 tiles, with the K split (and its fixup pass) for
//                    grids too small to fill the GPU and for operands past 2 GiB.
// launch_gemm picks the tile per launch from the row count (on the device when only the device
// knows it: k_gemm_bf16_pick runs the chosen kernel's blocks). In every kernel the
// accumulator tile is staged through LDS so the epilogues can pair columns (rotary halves,
// gate/up) and write coalesced rows. fp32 path (small models): 32x128x32 VALU tiles, same
// epilogues.
#include <algorithm>
#include <type_traits>

#include "kernels.h"

namespace akvs {

// g * sigmoid(g) with the hardware reciprocal (v_rcp_f32, 1 ulp) in place of an IEEE
// division, which cost about twice the instructions of the rest of the SwiGLU epilogue
__device__ __forceinline__ float silu(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
}

// Epilogue over an LDS tile Cs[BM][ldc] holding C[m0.., n0..] (SWIGLU: gate cols [0,BN/2),
// up cols [BN/2,BN) of output columns n0..n0+BN/2). Thread tid takes items tid + it * NT.
// The items go in groups whose loads (residual rows, row positions, rotary rows, LDS) are
// all issued before the group's first result is formed: one memory round trip per group
// instead of one per item (a loop over single items waits for every residual load, since
// the compiler cannot move it above the previous item's store to the same buffer).
template <int BM, int BN, int NT>
__device__ void epilogue_tile(const float *Cs, int ldc, int m0, int n0, int M_eff, int N,
                              const Epi &e) {
  // (loads go to clamped, in-bounds addresses whether or not their item is live, so that no
  // load sits in a branch whose join would wait for it; only the stores are conditional.
  // The thread index passes through an opaque move so that the item indices are formed
  // afresh in each call, not kept live from one half tile's epilogue to the next.)
  int tid;
  asm volatile("v_mov_b32 %0, %1" : "=v"(tid) : "v"((int)threadIdx.x));
  if (e.mode == EPI_STORE || e.mode == EPI_RESID) {
    constexpr int U = BN / 4, ITEMS = BM * U, IT = (ITEMS + NT - 1) / NT;
    constexpr int EG = IT < 8 ? IT : 8;
    const bool resid = e.mode == EPI_RESID;
    for (int it0 = 0; it0 < IT; it0 += EG) {
      __builtin_amdgcn_sched_barrier(0);  // one group's registers at a time
      float4 c[EG], h[EG];
#pragma unroll
      for (int j = 0; j < EG; ++j) {
        const int idx = min(tid + (it0 + j) * NT, ITEMS - 1);
        const int r = idx / U, c4 = (idx - r * U) * 4;
        c[j] = *reinterpret_cast<const float4 *>(Cs + r * ldc + c4);
        if (resid)  // N (the model width) is a multiple of 4 here
          h[j] = *reinterpret_cast<const float4 *>(
              reinterpret_cast<const float *>(e.out) +
              (size_t)min(m0 + r, M_eff - 1) * e.ldo + min(n0 + c4, N - 4));
      }
#pragma unroll
      for (int j = 0; j < EG; ++j) {
        const int idx = tid + (it0 + j) * NT;
        const int r = idx / U, c4 = (idx - r * U) * 4;
        const int gm = m0 + r, gn = n0 + c4;
        if (!(it0 + j < IT && idx < ITEMS && gm < M_eff && gn < N)) continue;
        const size_t off = (size_t)gm * e.ldo + gn;
        if (resid) {
          float4 v = h[j];
          v.x += c[j].x; v.y += c[j].y; v.z += c[j].z; v.w += c[j].w;
          *reinterpret_cast<float4 *>(reinterpret_cast<float *>(e.out) + off) = v;
        } else if (e.out_dtype == AKVS_BF16) {
          store4(reinterpret_cast<bf16_t *>(e.out) + off, c[j].x, c[j].y, c[j].z, c[j].w);
        } else {
          store4(reinterpret_cast<float *>(e.out) + off, c[j].x, c[j].y, c[j].z, c[j].w);
        }
      }
    }
  } else if (e.mode == EPI_SWIGLU) {
    constexpr int HALF = BN / 2, U = HALF / 4, ITEMS = BM * U, IT = (ITEMS + NT - 1) / NT;
    constexpr int EG = IT < 4 ? IT : 4;
    for (int it0 = 0; it0 < IT; it0 += EG) {
      __builtin_amdgcn_sched_barrier(0);  // one group's registers at a time
      float4 g[EG], u[EG];
#pragma unroll
      for (int j = 0; j < EG; ++j) {
        const int idx = min(tid + (it0 + j) * NT, ITEMS - 1);
        const int r = idx / U, c4 = (idx - r * U) * 4;
        g[j] = *reinterpret_cast<const float4 *>(Cs + r * ldc + c4);
        u[j] = *reinterpret_cast<const float4 *>(Cs + r * ldc + c4 + HALF);
      }
#pragma unroll
      for (int j = 0; j < EG; ++j) {
        const int idx = tid + (it0 + j) * NT;
        const int r = idx / U, c4 = (idx - r * U) * 4;
        const int gm = m0 + r, gn = n0 + c4;
        if (!(it0 + j < IT && idx < ITEMS && gm < M_eff && gn < N)) continue;
        const float a0 = silu(g[j].x) * u[j].x, a1 = silu(g[j].y) * u[j].y;
        const float a2 = silu(g[j].z) * u[j].z, a3 = silu(g[j].w) * u[j].w;
        if (e.out_dtype == AKVS_BF16)
          store4(reinterpret_cast<bf16_t *>(e.out) + (size_t)gm * e.ldo + gn, a0, a1, a2, a3);
        else
          store4(reinterpret_cast<float *>(e.out) + (size_t)gm * e.ldo + gn, a0, a1, a2, a3);
      }
    }
  } else {  // EPI_QKV: every tile holds whole heads of one section
    // hd (64 or 128) divides BN: a row holds BN / hd heads of hd / 8 items (4 columns of
    // each rotary half)
    const int hd = e.hd, half = hd >> 1;
    const int lu_shift = hd == 128 ? 4 : 3;  // log2 of the items per head (hd / 8)
    constexpr int items = BN / 8;
    constexpr int IT = (BM * items + NT - 1) / NT, EG = IT < 4 ? IT : 4;
    const float2 *rope = reinterpret_cast<const float2 *>(e.rope);
    int rpos[IT];  // row positions of this thread's items, all requested first
    if (e.pos) {
#pragma unroll
      for (int it = 0; it < IT; ++it)
        rpos[it] = e.pos[min(m0 + min((tid + it * NT) / items, BM - 1), M_eff - 1)];
    } else {
#pragma unroll
      for (int it = 0; it < IT; ++it) rpos[it] = e.pos0 + m0 + (tid + it * NT) / items;
    }
#pragma unroll
    for (int it0 = 0; it0 < IT; it0 += EG) {
      __builtin_amdgcn_sched_barrier(0);  // one group's registers at a time
      float lo[EG][4], hi[EG][4];
      float2 cs[EG][4];
#pragma unroll
      for (int j = 0; j < EG; ++j) {
        const int idx = min(tid + (it0 + j) * NT, BM * items - 1);
        const int r = idx / items, it_ = idx - r * items;
        const int hs = it_ >> lu_shift, u = it_ - (hs << lu_shift);
        const float *src = Cs + r * ldc + hs * hd + u * 4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          lo[j][i] = src[i];
          hi[j][i] = src[half + i];
        }
        if (rope) {
          const int p = min(max(rpos[it0 + j] - e.rope_base, 0), e.rope_rows - 1);
          const float2 *rr = rope + (size_t)p * half + u * 4;
#pragma unroll
          for (int i = 0; i < 4; ++i) cs[j][i] = rr[i];
        }
      }
#pragma unroll
      for (int j = 0; j < EG; ++j) {
        const int it = it0 + j;
        const int idx = tid + it * NT;
        const int r = idx / items, it_ = idx - r * items;
        const int hs = it_ >> lu_shift, u = it_ - (hs << lu_shift);
        const int gm = m0 + r;
        if (!(it < IT && idx < BM * items && gm < M_eff && n0 + hs * hd < N)) continue;
        const int col = e.n_off + n0 + hs * hd + u * 4;  // logical q|k|v column of the lo half
        if (col < e.hq_w + e.kv_w) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float a = lo[j][i], b = hi[j][i];
            lo[j][i] = a * cs[j][i].x - b * cs[j][i].y;
            hi[j][i] = b * cs[j][i].x + a * cs[j][i].y;
          }
        }
        size_t off;
        void *base;
        if (col < e.hq_w) {
          base = e.q_out;
          off = (size_t)gm * e.hq_w + col;
        } else {
          const int drow = e.kv_by_pos ? rpos[it] : gm;
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
          store4(d, lo[j][0], lo[j][1], lo[j][2], lo[j][3]);
          store4(d + half, hi[j][0], hi[j][1], hi[j][2], hi[j][3]);
        } else {
          float *d = reinterpret_cast<float *>(base) + off;
          store4(d, lo[j][0], lo[j][1], lo[j][2], lo[j][3]);
          store4(d + half, hi[j][0], hi[j][1], hi[j][2], hi[j][3]);
        }
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

// ------------------------------------------------------------------------------------------
// bf16 MFMA GEMM with 8 waves: 512-thread blocks (two waves per SIMD) on BM x BN x 64 block
// tiles, BM in {192, 256}, BN in {128, 256}. Waves form WGM x (8 / WGM), each owning
// (BM / WGM) x (BN * WGM / 8) outputs as v_mfma_f32_32x32x16_bf16 tiles. Against 128x128
// tiles of four waves this halves the operand bytes per flop while keeping two waves per
// SIMD. Operands arrive through buffer loads into NST register stages; each k-tile's LDS
// stores and global refills are spread over its four k-steps between the MFMAs
// (scheduling groups), so every wait before an LDS store covers only loads issued a tile
// earlier. The accumulators go through LDS half a tile of rows at a time for the shared
// epilogues. Rows past the device-side M are skipped, operand rows past M / N are clamped
// to valid rows (their results are discarded). The B row count (2N for SWIGLU) arrives as a
// kernel argument: derived on the device from the epilogue mode, the compiler keeps it in a
// vector register and wraps every B load in a loop over distinct descriptors.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t gemm_rsrc(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes,
                                           0x00020000);
}


// Output tile of block b: blocks past the live tile count exit; the live blocks are spread
// so that each XCD (blocks b, b+8, ... of the dispatch order) takes one contiguous run of
// the logical tile order, and the logical order walks groups of GM row tiles, rows fastest,
// so that the blocks resident on one XCD share a few A and B panels in its L2.
template <int GM>
__device__ __forceinline__ bool grouped_tile(int b, int m_tiles, int n_tiles, int &mt, int &nt) {
  const int live = m_tiles * n_tiles;
  if (b >= live) return false;
  const int x = b & 7, idx = b >> 3;
  const int base = live >> 3, extra = live & 7;
  const int t = x * base + min(x, extra) + idx;
  const int per_group = GM * n_tiles;
  const int g = t / per_group, local = t - g * per_group;
  const int rows = min(GM, m_tiles - g * GM);
  mt = g * GM + local % rows;
  nt = local / rows;
  return true;
}

template <int BM, int BN, int WGM, int NST>
struct Gemm8 {
  static constexpr int WGN = 8 / WGM, WM = BM / WGM, WN = BN / WGN;
  static constexpr int MI = WM / 32, NJ = WN / 32;
  static constexpr int ACH = BM / 64, BCH = BN / 64, CH = ACH + BCH;  // 16-B chunks per thread
  static constexpr int ATILE = BM * G_LDS, BUF = (BM + BN) * G_LDS;  // bf16 elements
  static constexpr int HB = BM / 2, CLD = BN + 4;                    // epilogue half tile
  static constexpr int LOOP_BYTES = 2 * BUF * 2, C_BYTES = HB * CLD * 4;
  static constexpr int SMEM = LOOP_BYTES > C_BYTES ? LOOP_BYTES : C_BYTES;
  static_assert(WGM == 2 || WGM == 4, "wave rows must split in two halves");
};

// Body of block `bid` of the 8-wave kernel on LDS `smem` (S::SMEM bytes), M_eff live rows.
// With splits > 1 block bid computes k-slice bid % splits of tile bid / splits and writes
// its fp32 partial tile to part ([tile][split][BM][BN], tiles in row-major order) for
// k_gemm_fixup, which adds the slices in order and runs the epilogue.
template <int BM, int BN, int WGM, int NST>
__device__ __forceinline__ void gemm_w8_body(unsigned char *smem, int bid,
                                             const bf16_t *__restrict__ A, int lda,
                                             const bf16_t *__restrict__ B, int ldb, int M_eff,
                                             int N, int K, int b_rows, const Epi &epi,
                                             int splits = 1, float *part = nullptr) {
  using S = Gemm8<BM, BN, WGM, NST>;
  bf16_t *sm = reinterpret_cast<bf16_t *>(smem);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / S::WGN, wn = wave % S::WGN;
  const bool swiglu = epi.mode == EPI_SWIGLU;
  const int bn_out = swiglu ? BN / 2 : BN;
  const int n_tiles = (N + bn_out - 1) / bn_out;
  const int tile_bid = bid / splits, split = bid - tile_bid * splits;
  int mt_, nt_;
  if (!grouped_tile<8>(tile_bid, (M_eff + BM - 1) / BM, n_tiles, mt_, nt_)) return;
  const int m0 = mt_ * BM;
  const int n0 = nt_ * bn_out;
  const __amdgpu_buffer_rsrc_t ra = gemm_rsrc(A, (uint32_t)((size_t)M_eff * lda * 2));
  const __amdgpu_buffer_rsrc_t rb = gemm_rsrc(B, (uint32_t)b_rows * (uint32_t)ldb * 2u);

  // chunk c of a thread: row (tid >> 3) + 64 c of the stacked [A tile; B tile], k columns
  // (tid & 7) * 8 ..+7; SWIGLU B tiles stack BN/2 gate rows over the matching up rows
  int goff[S::CH], loff[S::CH];
#pragma unroll
  for (int c = 0; c < S::CH; ++c) {
    const int r = (tid >> 3) + 64 * c, kc = (tid & 7) * 8;
    if (c < S::ACH) {
      goff[c] = (min(m0 + r, M_eff - 1) * lda + kc) * 2;
    } else {
      const int rb_ = r - BM;
      int gn;
      if (swiglu) {
        const int oc = min(n0 + (rb_ & (BN / 2 - 1)), N - 1);
        gn = rb_ < BN / 2 ? oc : N + oc;
      } else {
        gn = min(n0 + rb_, N - 1);
      }
      goff[c] = (gn * ldb + kc) * 2;
    }
    loff[c] = r * G_LDS + kc;
  }
  const int nk_all = K / GB_K;
  const int per = (nk_all + splits - 1) / splits;
  const int kt0 = min(nk_all, split * per);
  const int nk = max(1, min(nk_all, kt0 + per) - kt0);  // >= 1: splits <= nk_all

  f32x16_t acc[S::MI][S::NJ];
#pragma unroll
  for (int i = 0; i < S::MI; ++i)
#pragma unroll
    for (int j = 0; j < S::NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  u32x4_t rg[NST][S::CH];
  bf16x8_t fa[2][S::MI], fb[2][S::NJ];
  const int fa_lane = (wm * S::WM + (lane & 31)) * G_LDS + (lane >> 5) * 8;
  const int fb_lane = S::ATILE + (wn * S::WN + (lane & 31)) * G_LDS + (lane >> 5) * 8;

#define AKVS_W8_GL(ST, KT, C0, C1)                                                          \
  {                                                                                         \
    const int so_ = (kt0 + (KT)) * GB_K * 2;                                                \
    _Pragma("unroll") for (int c = (C0); c < (C1); ++c) rg[ST][c] = __builtin_bit_cast(     \
        u32x4_t, c < S::ACH ? __builtin_amdgcn_raw_buffer_load_b128(ra, goff[c], so_, 0)    \
                            : __builtin_amdgcn_raw_buffer_load_b128(rb, goff[c], so_, 0));  \
  }
#define AKVS_W8_SS(ST, BOFF, C0, C1)                                                        \
  {                                                                                         \
    bf16_t *b_ = sm + (BOFF);                                                               \
    _Pragma("unroll") for (int c = (C0); c < (C1); ++c)                                     \
        *reinterpret_cast<u32x4_t *>(b_ + loff[c]) = rg[ST][c];                             \
  }
#define AKVS_W8_FR(F, BOFF, KS)                                                             \
  {                                                                                         \
    const bf16_t *As_ = sm + (BOFF) + fa_lane + (KS) * 16;                                  \
    const bf16_t *Bs_ = sm + (BOFF) + fb_lane + (KS) * 16;                                  \
    _Pragma("unroll") for (int i = 0; i < S::MI; ++i) fa[F][i] =                            \
        *reinterpret_cast<const bf16x8_t *>(As_ + i * 32 * G_LDS);                          \
    _Pragma("unroll") for (int j = 0; j < S::NJ; ++j) fb[F][j] =                            \
        *reinterpret_cast<const bf16x8_t *>(Bs_ + j * 32 * G_LDS);                          \
  }
  // k-tile T from LDS buffer `cur`; ring slot P holds tile T+1, which goes to buffer `nxt`
  // a quarter per k-step while the slot refills with tile T+NST+1 (loads past the range
  // re-read the last tile, so every load is unconditional and the waits stay exact)
#define AKVS_W8_ITER(T, P)                                                                  \
  {                                                                                         \
    AKVS_W8_FR(0, cur, 0);                                                                  \
    _Pragma("unroll") for (int ks = 0; ks < 4; ++ks) {                                      \
      if (ks < 3) AKVS_W8_FR((ks + 1) & 1, cur, ks + 1);                                    \
      const int q0_ = ks * S::CH / 4, q1_ = (ks + 1) * S::CH / 4;                           \
      AKVS_W8_SS(P, nxt, q0_, q1_);                                                         \
      AKVS_W8_GL(P, min((T) + NST + 1, nk - 1), q0_, q1_);                                  \
      _Pragma("unroll") for (int i = 0; i < S::MI; ++i)                                     \
          _Pragma("unroll") for (int j = 0; j < S::NJ; ++j) acc[i][j] =                     \
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ks & 1][i], fb[ks & 1][j],         \
                                                      acc[i][j], 0, 0, 0);                  \
      _Pragma("unroll") for (int g_ = 0; g_ < S::MI * S::NJ; ++g_) {                        \
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                  \
        if (ks < 3 && g_ < S::MI + S::NJ) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0); \
        if (g_ < q1_ - q0_) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);              \
        if (g_ >= (S::MI * S::NJ) / 2 && g_ < (S::MI * S::NJ) / 2 + (q1_ - q0_))            \
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                                \
      }                                                                                     \
      __builtin_amdgcn_sched_barrier(0);                                                    \
    }                                                                                       \
    __syncthreads();                                                                        \
    {                                                                                       \
      const int t_ = cur;                                                                   \
      cur = nxt;                                                                            \
      nxt = t_;                                                                             \
    }                                                                                       \
  }
  int cur = 0, nxt = S::BUF;
  AKVS_W8_GL(0, 0, 0, S::CH);
  AKVS_W8_SS(0, 0, 0, S::CH);
#pragma unroll
  for (int st = 0; st < NST; ++st) AKVS_W8_GL(st, min(1 + st, nk - 1), 0, S::CH);
  __syncthreads();
  int t = 0;
  if (NST == 1) {
    for (; t < nk; ++t) AKVS_W8_ITER(t, 0);
  } else {
    for (; t + 2 <= nk; t += 2) {
      AKVS_W8_ITER(t, 0);
      AKVS_W8_ITER(t + 1, NST - 1);
    }
    if (t < nk) AKVS_W8_ITER(t, 0);
  }
#undef AKVS_W8_ITER
#undef AKVS_W8_FR
#undef AKVS_W8_SS
#undef AKVS_W8_GL

  if (splits > 1) {  // this k-slice's fp32 partial tile, rows of BN floats
    const int t_rm = mt_ * n_tiles + nt_;
    float *dst = part + ((size_t)t_rm * splits + split) * BM * BN;
#pragma unroll
    for (int i = 0; i < S::MI; ++i)
#pragma unroll
      for (int j = 0; j < S::NJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wm * S::WM + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
          const int col = wn * S::WN + j * 32 + (lane & 31);
          dst[row * BN + col] = acc[i][j][r];
        }
    return;
  }

  // epilogue: rows [h * HB, (h + 1) * HB) of the tile belong to waves wm / (WGM / 2) == h
  float *Cs = reinterpret_cast<float *>(smem);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (m0 + h * S::HB >= M_eff) break;  // block-uniform
    if (wm / (WGM / 2) == h) {
#pragma unroll
      for (int i = 0; i < S::MI; ++i)
#pragma unroll
        for (int j = 0; j < S::NJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = wm * S::WM - h * S::HB + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 +
                            (r & 3);
            const int col = wn * S::WN + j * 32 + (lane & 31);
            Cs[row * S::CLD + col] = acc[i][j][r];
          }
    }
    __syncthreads();
    epilogue_tile<S::HB, BN, 512>(Cs, S::CLD, m0 + h * S::HB, n0, M_eff, N, epi);
    __syncthreads();
  }
}

template <int BM, int BN, int WGM, int NST>
__global__ __launch_bounds__(512, 1) void k_gemm_bf16_w8(const bf16_t *__restrict__ A, int lda,
                                                         const bf16_t *__restrict__ B, int ldb,
                                                         int M, int N, int K, int b_rows,
                                                         const int32_t *m_dev, Epi epi) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[Gemm8<BM, BN, WGM, NST>::SMEM];
  const int M_eff = m_dev ? min(M, *m_dev) : M;
  gemm_w8_body<BM, BN, WGM, NST>(smem, blockIdx.x, A, lda, B, ldb, M_eff, N, K, b_rows, epi);
}

// ------------------------------------------------------------------------------------------
// bf16 MFMA GEMM, 8 waves in two groups that take turns ("ping-pong"). Waves w and w + 4 of
// a block run on the same SIMD, so group 0 (waves 0-3) and group 1 (waves 4-7) hold one wave
// of every SIMD. Group g owns rows [g BM/2, (g+1) BM/2) of the BM x BN block tile, as four
// waves side by side over BN, each (BM/2) x (BN/4) in 32x32 MFMA tiles. The two groups run
// half a k-tile apart and alternate two phases, each closed by a block barrier:
//   memory phase of k-tile t: read all of this wave's operand fragments of tile t from LDS
//     into registers, store this thread's share of tile t+1 (loaded two phases earlier)
//     into the other LDS buffer, and issue the global loads of its share of tile t+2;
//   compute phase of k-tile t: only the MFMAs over the fragments already in registers.
// So while one wave of a SIMD multiplies, the other feeds LDS and memory, and the MFMA pipe
// is never left waiting on a wave's own loads. Group 1 starts one phase late and finishes
// one phase late; both groups pass the same number of barriers. Buffer hazards: tile t+1 is
// written into the buffer of tile t-1 only after both groups read tile t-1 (the barrier
// before the writing phase follows the second group's reads, which complete before it).
template <int BM, int BN>
struct GemmPP {
  static constexpr int HM = BM / 2, WM = HM, WN = BN / 4;
  static constexpr int MI = WM / 32, NJ = WN / 32;
  static constexpr int CH = (BM + BN) / 64;  // 16-byte chunks per thread per k-tile
  static constexpr int ACH = BM / 64;
  static constexpr int ATILE = BM * G_LDS, BUF = (BM + BN) * G_LDS;
  static constexpr int CLD = BN + 4;
  static constexpr int LOOP_BYTES = 2 * BUF * 2, C_BYTES = HM * CLD * 4;
  static constexpr int SMEM = LOOP_BYTES > C_BYTES ? LOOP_BYTES : C_BYTES;
  static_assert(BM % 64 == 0 && WM % 32 == 0 && WN % 32 == 0, "tile shape");
};

template <int BM, int BN>
__device__ __forceinline__ void gemm_pp_body(unsigned char *smem, int bid,
                                             const bf16_t *__restrict__ A, int lda,
                                             const bf16_t *__restrict__ B, int ldb, int M_eff,
                                             int N, int K, int b_rows, const Epi &epi) {
  using S = GemmPP<BM, BN>;
  bf16_t *sm = reinterpret_cast<bf16_t *>(smem);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = wave >> 2, wn = wave & 3;
  const bool swiglu = epi.mode == EPI_SWIGLU;
  const int bn_out = swiglu ? BN / 2 : BN;
  const int n_tiles = (N + bn_out - 1) / bn_out;
  int mt_, nt_;
  if (!grouped_tile<8>(bid, (M_eff + BM - 1) / BM, n_tiles, mt_, nt_)) return;
  const int m0 = mt_ * BM;
  const int n0 = nt_ * bn_out;
  const __amdgpu_buffer_rsrc_t ra = gemm_rsrc(A, (uint32_t)((size_t)M_eff * lda * 2));
  const __amdgpu_buffer_rsrc_t rb = gemm_rsrc(B, (uint32_t)b_rows * (uint32_t)ldb * 2u);

  // chunk c of a thread: row (tid >> 3) + 64 c of the stacked [A tile; B tile], k columns
  // (tid & 7) * 8 ..+7 (the same map as the 8-wave kernel, SWIGLU stacking included)
  int goff[S::CH], loff[S::CH];
#pragma unroll
  for (int c = 0; c < S::CH; ++c) {
    const int r = (tid >> 3) + 64 * c, kc = (tid & 7) * 8;
    if (c < S::ACH) {
      goff[c] = (min(m0 + r, M_eff - 1) * lda + kc) * 2;
    } else {
      const int rb_ = r - BM;
      int gn;
      if (swiglu) {
        const int oc = min(n0 + (rb_ & (BN / 2 - 1)), N - 1);
        gn = rb_ < BN / 2 ? oc : N + oc;
      } else {
        gn = min(n0 + rb_, N - 1);
      }
      goff[c] = (gn * ldb + kc) * 2;
    }
    loff[c] = r * G_LDS + kc;
  }
  const int nk = K / GB_K;

  f32x16_t acc[S::MI][S::NJ];
#pragma unroll
  for (int i = 0; i < S::MI; ++i)
#pragma unroll
    for (int j = 0; j < S::NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  u32x4_t rg[S::CH];
  bf16x8_t fa[4][S::MI], fb[4][S::NJ];
  const int fa_lane = (grp * S::HM + (lane & 31)) * G_LDS + (lane >> 5) * 8;
  const int fb_lane = S::ATILE + (wn * S::WN + (lane & 31)) * G_LDS + (lane >> 5) * 8;

  auto gload = [&](int kt) {
    const int so = kt * GB_K * 2;
#pragma unroll
    for (int c = 0; c < S::CH; ++c)
      rg[c] = __builtin_bit_cast(u32x4_t,
                                 c < S::ACH ? __builtin_amdgcn_raw_buffer_load_b128(ra, goff[c], so, 0)
                                            : __builtin_amdgcn_raw_buffer_load_b128(rb, goff[c], so, 0));
  };
  auto lstore = [&](int boff) {
#pragma unroll
    for (int c = 0; c < S::CH; ++c) *reinterpret_cast<u32x4_t *>(sm + boff + loff[c]) = rg[c];
  };
  auto fread = [&](int boff) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int i = 0; i < S::MI; ++i)
        fa[ks][i] = *reinterpret_cast<const bf16x8_t *>(sm + boff + fa_lane + i * 32 * G_LDS + ks * 16);
#pragma unroll
      for (int j = 0; j < S::NJ; ++j)
        fb[ks][j] = *reinterpret_cast<const bf16x8_t *>(sm + boff + fb_lane + j * 32 * G_LDS + ks * 16);
    }
  };

  gload(0);
  lstore(0);
  if (nk > 1) gload(1);
  __syncthreads();
  if (grp == 1) __syncthreads();  // group 1 starts one phase late
  for (int t = 0; t < nk; ++t) {
    const int cur = (t & 1) * S::BUF, nxt = S::BUF - cur;
    fread(cur);
    if (t + 1 < nk) lstore(nxt);
    if (t + 2 < nk) gload(t + 2);
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int i = 0; i < S::MI; ++i)
#pragma unroll
        for (int j = 0; j < S::NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ks][i], fb[ks][j], acc[i][j], 0, 0, 0);
    if (grp == 0 || t + 1 < nk) __syncthreads();  // group 1 skips its last one
  }
  __syncthreads();

  // epilogue: half h of the tile's rows is group h's
  float *Cs = reinterpret_cast<float *>(smem);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (m0 + h * S::HM >= M_eff) break;  // block-uniform
    if (grp == h) {
#pragma unroll
      for (int i = 0; i < S::MI; ++i)
#pragma unroll
        for (int j = 0; j < S::NJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            const int col = wn * S::WN + j * 32 + (lane & 31);
            Cs[row * S::CLD + col] = acc[i][j][r];
          }
    }
    __syncthreads();
    epilogue_tile<S::HM, BN, 512>(Cs, S::CLD, m0 + h * S::HM, n0, M_eff, N, epi);
    __syncthreads();
  }
}

template <int BM, int BN>
__global__ __launch_bounds__(512, 1) void k_gemm_bf16_pp(const bf16_t *__restrict__ A, int lda,
                                                         const bf16_t *__restrict__ B, int ldb,
                                                         int M, int N, int K, int b_rows,
                                                         const int32_t *m_dev, Epi epi) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[GemmPP<BM, BN>::SMEM];
  const int M_eff = m_dev ? min(M, *m_dev) : M;
  gemm_pp_body<BM, BN>(smem, blockIdx.x, A, lda, B, ldb, M_eff, N, K, b_rows, epi);
}

// Block tiles of the 8-wave kernels with their rate per CU relative to the 256x256 tile,
// measured on the 3B projection shapes with every CU busy (M = 1405 and 4516 rows). A launch
// takes the tile with the least (rounds of one tile per CU) x (tile area) / rate at its row
// count. The ping-pong kernel needs long compute phases: only its 192x256 tile was kept
// (with 128 columns per tile a phase holds 12 MFMAs and the shared schedule is faster; at
// 192x256 the shared schedule measured 0.75 against the ping-pong's 0.88). Checked on the
// 7B and 32B projection shapes with the clocks warmed up: the model's pick was the fastest
// tile or within a few percent of it.
struct W8Tile {
  int bm, bn;
  bool pp;
  float rate;
};
constexpr int kW8Count = 4;
__host__ __device__ inline W8Tile w8_tile(int i) {
  switch (i) {
    case 0: return {256, 256, false, 1.0f};
    case 1: return {192, 256, true, 0.88f};
    case 2: return {256, 128, false, 0.78f};
    default: return {192, 128, false, 0.74f};
  }
}
__host__ __device__ inline int gemm_w8_tile(int M, int N, int mode, int cus) {
  int best = 0;
  float best_cost = 0;
  for (int i = 0; i < kW8Count; ++i) {
    const W8Tile c = w8_tile(i);
    const int bn_out = mode == EPI_SWIGLU ? c.bn / 2 : c.bn;
    const int tiles = ((M + c.bm - 1) / c.bm) * ((N + bn_out - 1) / bn_out);
    const float cost = (float)((tiles + cus - 1) / cus) * (float)(c.bm * c.bn) / c.rate;
    if (i == 0 || cost < best_cost) {
      best = i;
      best_cost = cost;
    }
  }
  return best;
}

// K split of the 192x128 8-wave tile for row counts whose tiles would leave at least half of
// the CUs idle (probe layers at small refresh ratios, the query rows of the last layer):
// about one round of (tile, k-slice) items, slices of at least 8 k-tiles, at most 12 per
// tile; k_gemm_fixup adds the slices in order. (At 810 rows of the 3B shape the output and
// down projections make 120 such tiles for 256 CUs; at 171 rows 24.)
constexpr int kW8SplitBM = 192, kW8SplitBN = 128;
__host__ __device__ inline int w8_k_splits(int M, int N, int K, int mode, int cus) {
  const int bn_out = mode == EPI_SWIGLU ? kW8SplitBN / 2 : kW8SplitBN;
  const int tiles = ((M + kW8SplitBM - 1) / kW8SplitBM) * ((N + bn_out - 1) / bn_out);
  const int nk = K / GB_K;
  if (tiles <= 0 || 2 * tiles > cus || nk < 32) return 1;
  int sp = cus / tiles;
  if (sp > nk / 8) sp = nk / 8;
  if (sp > 12) sp = 12;
  return sp < 2 ? 1 : sp;
}

// One launch for a row count known only on the device: each block applies the tile model
// (and, with a partial-tile workspace, the K split) to the live row count and runs as a
// block of the chosen kernel (blocks past that kernel's item count exit). The grid covers
// the largest of the grids over the row counts the host cannot rule out.
constexpr int kPickSmem =
    std::max(std::max(Gemm8<256, 256, 2, 1>::SMEM, GemmPP<192, 256>::SMEM),
             std::max(Gemm8<256, 128, 4, 2>::SMEM, Gemm8<192, 128, 2, 2>::SMEM));
__global__ __launch_bounds__(512, 1) void k_gemm_bf16_pick(const bf16_t *__restrict__ A, int lda,
                                                           const bf16_t *__restrict__ B, int ldb,
                                                           int M, int N, int K, int b_rows,
                                                           const int32_t *m_dev, Epi epi,
                                                           int cus, float *part) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[kPickSmem];
  const int M_eff = m_dev ? min(M, *m_dev) : M;
  const int sp = part ? w8_k_splits(M_eff, N, K, epi.mode, cus) : 1;
  if (sp > 1) {
    gemm_w8_body<kW8SplitBM, kW8SplitBN, 2, 2>(smem, blockIdx.x, A, lda, B, ldb, M_eff, N, K,
                                               b_rows, epi, sp, part);
    return;
  }
  switch (gemm_w8_tile(M_eff, N, epi.mode, cus)) {
    case 0:
      gemm_w8_body<256, 256, 2, 1>(smem, blockIdx.x, A, lda, B, ldb, M_eff, N, K, b_rows, epi);
      break;
    case 1:
      gemm_pp_body<192, 256>(smem, blockIdx.x, A, lda, B, ldb, M_eff, N, K, b_rows, epi);
      break;
    case 2:
      gemm_w8_body<256, 128, 4, 2>(smem, blockIdx.x, A, lda, B, ldb, M_eff, N, K, b_rows, epi);
      break;
    default:
      gemm_w8_body<192, 128, 2, 2>(smem, blockIdx.x, A, lda, B, ldb, M_eff, N, K, b_rows, epi);
      break;
  }
}

// Sum of n partial float4s p[0], p[stride], ... added in index order; eight loads are in
// flight before their adds, so the pass costs about n / 8 memory round trips.
__device__ __forceinline__ float4 sum_pieces(const float *p, size_t stride, int n) {
  float4 acc = *reinterpret_cast<const float4 *>(p);
  int k = 1;
  for (; k + 8 <= n; k += 8) {
    float4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = *reinterpret_cast<const float4 *>(p + (size_t)(k + u) * stride);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      acc.x += v[u].x; acc.y += v[u].y; acc.z += v[u].z; acc.w += v[u].w;
    }
  }
  for (; k < n; ++k) {
    const float4 v = *reinterpret_cast<const float4 *>(p + (size_t)k * stride);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  return acc;
}

// Second pass of a K-split GEMM: a block takes G_FR rows of one tile, adds their partial
// rows in split order into an LDS slice and runs the epilogue on it.
constexpr int G_FR = 16;
// W8: partials of the 192x128 8-wave tile (split by w8_k_splits, n_slots = CU count), else
// of the 4-wave 128x128 kernel (gemm_k_splits).
template <int BM, bool W8>
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
  const int splits = W8 ? w8_k_splits(M_eff, N, K, epi.mode, n_slots)
                        : gemm_k_splits(tiles, K / GB_K, n_slots);
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
    const float4 acc = sum_pieces(src + row * GB_N + c4, (size_t)BM * GB_N, splits);
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
  size_t floats = items * 128 * GB_N;
  // the 8-wave split: at most one (tile, slice) item per CU, for any row count up to M
  const int cus = gemm_cu_count();
  for (int m = 1; m <= M; m = (m == M ? M + 1 : std::min(M, m + 16))) {
    if (w8_k_splits(m, N, K, mode, cus) > 1) {
      floats = std::max(floats, (size_t)cus * kW8SplitBM * kW8SplitBN);
      break;
    }
  }
  return floats;
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

template <int BM, int BN, int WGM, int NST>
static void launch_w8(const void *A, int lda, const void *B, int ldb, int M, int N, int K,
                      const int32_t *m_dev, const Epi &epi, hipStream_t s) {
  const int bn_out = epi.mode == EPI_SWIGLU ? BN / 2 : BN;
  const int grid = ((M + BM - 1) / BM) * ((N + bn_out - 1) / bn_out);
  hipLaunchKernelGGL((k_gemm_bf16_w8<BM, BN, WGM, NST>), dim3(grid), dim3(512), 0, s,
                     reinterpret_cast<const bf16_t *>(A), lda,
                     reinterpret_cast<const bf16_t *>(B), ldb, M, N, K,
                     epi.mode == EPI_SWIGLU ? 2 * N : N, m_dev, epi);
}

template <int BM, int BN>
static void launch_pp(const void *A, int lda, const void *B, int ldb, int M, int N, int K,
                      const int32_t *m_dev, const Epi &epi, hipStream_t s) {
  const int bn_out = epi.mode == EPI_SWIGLU ? BN / 2 : BN;
  const int grid = ((M + BM - 1) / BM) * ((N + bn_out - 1) / bn_out);
  hipLaunchKernelGGL((k_gemm_bf16_pp<BM, BN>), dim3(grid), dim3(512), 0, s,
                     reinterpret_cast<const bf16_t *>(A), lda,
                     reinterpret_cast<const bf16_t *>(B), ldb, M, N, K,
                     epi.mode == EPI_SWIGLU ? 2 * N : N, m_dev, epi);
}

// The 8-wave launch for one row-count range: the tile (and K split) every count in
// [lo, M] picks, or -1 when they differ (the device then picks); any_split when some count
// in the range splits K.
struct W8Choice {
  int choice;  // kernel index of w8_tile, 100 + splits for the split 192x128 tile, -1 mixed
  bool any_split;
};
static W8Choice w8_choice(int M, int N, int K, const int32_t *m_dev, int mode,
                          const float *part, int m_min) {
  const int cus = gemm_cu_count();
  auto at = [&](int m) {
    const int sp = part ? w8_k_splits(m, N, K, mode, cus) : 1;
    return sp > 1 ? 100 + sp : gemm_w8_tile(m, N, mode, cus);
  };
  W8Choice c{at(M), false};
  c.any_split = c.choice >= 100;
  if (m_dev) {
    for (int m = std::max(m_min, 1); m < M; m = std::min(M, m + 16)) {
      const int x = at(m);
      c.any_split |= x >= 100;
      if (x != c.choice) c.choice = -1;
    }
  }
  if (c.any_split) c.choice = -1;  // the split launches go through the picking kernel
  return c;
}

hipError_t launch_gemm(const void *A, int lda, const void *B, int ldb, int M, int N, int K,
                       const int32_t *m_dev, int dtype, const Epi &epi, hipStream_t s,
                       float *part, int m_min) {
  if (M == 0 || N == 0) return hipSuccess;
  if (dtype == AKVS_BF16) {
    const size_t b_rows = epi.mode == EPI_SWIGLU ? 2 * (size_t)N : (size_t)N;
    // buffer offsets are 32-bit: larger operands stay on the 4-wave kernel
    const bool fits = (size_t)M * lda * 2 < (1u << 31) && b_rows * ldb * 2 < (1u << 31);
    if (fits) {
      const int cus = gemm_cu_count();
      const W8Choice c = w8_choice(M, N, K, m_dev, epi.mode, part, m_min);
      if (c.choice < 0) {
        int grid = c.any_split ? cus : 0;
        for (int i = 0; i < kW8Count; ++i) {
          const W8Tile t = w8_tile(i);
          const int bn_out = epi.mode == EPI_SWIGLU ? t.bn / 2 : t.bn;
          grid = std::max(grid, ((M + t.bm - 1) / t.bm) * ((N + bn_out - 1) / bn_out));
        }
        hipLaunchKernelGGL(k_gemm_bf16_pick, dim3(grid), dim3(512), 0, s,
                           reinterpret_cast<const bf16_t *>(A), lda,
                           reinterpret_cast<const bf16_t *>(B), ldb, M, N, K,
                           epi.mode == EPI_SWIGLU ? 2 * N : N, m_dev, epi, cus,
                           c.any_split ? part : nullptr);
        return hipGetLastError();
      }
      switch (c.choice) {
        case 0: launch_w8<256, 256, 2, 1>(A, lda, B, ldb, M, N, K, m_dev, epi, s); break;
        case 1: launch_pp<192, 256>(A, lda, B, ldb, M, N, K, m_dev, epi, s); break;
        case 2: launch_w8<256, 128, 4, 2>(A, lda, B, ldb, M, N, K, m_dev, epi, s); break;
        default: launch_w8<192, 128, 2, 2>(A, lda, B, ldb, M, N, K, m_dev, epi, s); break;
      }
      return hipGetLastError();
    }
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

hipError_t launch_gemm_fixup(const void *, int lda, const void *, int ldb, int M, int N, int K,
                             const int32_t *m_dev, int dtype, const Epi &epi, hipStream_t s,
                             float *part, int m_min) {
  if (M == 0 || N == 0 || dtype != AKVS_BF16) return hipSuccess;
  const size_t b_rows = epi.mode == EPI_SWIGLU ? 2 * (size_t)N : (size_t)N;
  const bool fits = (size_t)M * lda * 2 < (1u << 31) && b_rows * ldb * 2 < (1u << 31);
  if (fits) {
    const W8Choice c = w8_choice(M, N, K, m_dev, epi.mode, part, m_min);
    if (!c.any_split) return hipSuccess;
    const int bn_out = epi.mode == EPI_SWIGLU ? kW8SplitBN / 2 : kW8SplitBN;
    const int tiles = ((M + kW8SplitBM - 1) / kW8SplitBM) * ((N + bn_out - 1) / bn_out);
    hipLaunchKernelGGL((k_gemm_fixup<kW8SplitBM, true>), dim3(tiles * (kW8SplitBM / G_FR)),
                       dim3(256), 0, s, M, N, K, m_dev, epi, gemm_cu_count(), part);
    return hipGetLastError();
  }
  const GemmPlan p = gemm_plan(M, N, K, m_dev, epi, part, m_min);
  if (!p.any_split) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_fixup<128, false>), dim3(p.tiles_cap * (128 / G_FR)), dim3(256), 0, s,
                     M, N, K, m_dev, epi, p.n_slots, part);
  return hipGetLastError();
}

}  // namespace akvs
