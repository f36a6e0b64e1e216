// Attention of (sparse, position-sorted) query rows over a causal key range.
//
// bf16 path: one block = a group of the query heads that read one KV head, over a tile of
// rows; each wave owns 32 rows of one query head. Keys stream through LDS in tiles of 64
// (K and V row-major), shared by every wave of the block. Scores are computed
// transposed, S^T = K Q^T, with MFMA 32x32x16 bf16: each lane then holds 16 scores of ONE
// query row (the other 16 of that row's 32 keys sit in lane ^ 32), and the probabilities
// already sit in the operand layout of the second product O^T = V^T P^T (the pairing of
// the 16 contraction slots with keys is a fixed permutation applied to both operands).
// The running maximum is only raised when a score exceeds it by more than 2^8, which
// keeps the rescaling of O off the common path while p = 2^(s - m) stays <= 256.
// Row tiles are launched longest-first (rows are sorted by position, so later tiles
// see more keys).
#include "kernels.h"

namespace akvs {

// V tile: 64 keys x hd, row-major as in memory, rows padded by 32 elements (64 bytes, a
// 16-bank shift per row). The P.V operand wants, per lane, 8 keys of ONE head dim; gfx950's
// transposing LDS read (ds_read_b64_tr_b16) delivers that from row-major rows: within
// each 16-lane group, lane j receives element j % 4 of the 8-byte chunk addressed by lane
// 4k + j / 4, for k = 0..3. So source lane s of a group points at key row +s/4, head dims
// 4*(s%4)..+3 of the group's 16 dims, and each lane gets 4 consecutive keys of its dim per
// read. Against the transposed V^T staging it replaced (VALU byte shuffles and 8-byte LDS
// stores in the loading waves), same bits: 1-4 % faster on the 32B, 7B and 3B shapes
// (standalone timing, not in the repository). A 32-lane read phase touches 4 rows x 64
// bytes, at 16-bank offsets: no conflicts.

// Block shape: one query head per block, 32-row waves. With about 250 VGPRs a compute unit
// holds eight waves, so blocks of 8 waves (one per unit) or 4 (two per unit) use every SIMD
// evenly; the first four waves stage the K / V tiles.
//  - 256 rows (8 waves sharing each K / V tile) when that still makes 512 blocks (32B probe
//    layer, 5527 rows over 16128 keys: 1094 us against 1383 us for blocks that grouped the
//    five query heads of a KV head over 32 rows, whose 5 waves leave SIMDs unevenly loaded);
//  - else 128 rows (4 waves) per block; when those make fewer than 512 blocks the key range
//    is split as well (see attn_splits). (32B probe layer at r = 1/10, 3050 rows: 664 us
//    against 751 us for the five-head 32-row blocks; the 3B full prefill measured the same
//    with three-head 64-row blocks. Grouped-head blocks never make more blocks than these,
//    so they are not used; the kernel still takes the general head grouping gh.)
struct AttnShape {
  int gh, n_groups, nrb;
};
static inline AttnShape attn_shape(int G, int rows, int hkv) {
  AttnShape a{0, 0, 0};
  if (G < 1) return a;
  a.gh = 1;
  a.n_groups = G;
  a.nrb = (long long)((rows + 255) / 256) * hkv * G >= 512 ? 8 : 4;
  return a;
}

// Planned split (launch_attention_plan, then launch_attention with the plan): for calls
// over few position-sorted rows, whose tiles leave block slots idle or end at very
// different times, the key range of each tile is cut into nearly equal pieces sized so
// that every block slot of the chip gets about the same work, and the pieces go out
// longest first. Block shape and item budget from the row bound (host):
//  - 4-wave 128-row blocks (two per CU) in one round, where the 128-row tiles fill at most
//    3/4 of the round's items (slots / heads) and are at least 3;
//  - else 8-wave 256-row blocks (one per CU): one round where their tiles fill at most
//    half of it, two rounds where they fill less than two;
//  - else no plan (the tiles alone fill the chip; launch_attention's own split applies).
// Measured on the 3B-class probe layers (1441 / 865 / 300 / 166 rows over 4516 keys):
// 75 / 53 / 38 / 35 us against 92 / 60 / 47 / 37 us; 7B-class (2802 / 1513 rows over
// 8128 keys) 199 / 129 against 215 / 155 us; the query rows of the last layer (64 over
// 4516 keys, 128 over 16128) 27 / 69 against 28 / 79 us. With one round for the 3B
// layers at 1992 rows over 4516 keys the 128-row blocks took 101 us against 89 us for two
// rounds of 256-row blocks, which is what sets the 3/4 bound (standalone harness, not in
// the repository).
struct AttnEqShape {
  int rb, budget, max_pc;
  bool use;
};
constexpr int kAttnMaxPieces = 8;  // the merge's all-at-once path
static inline AttnEqShape attn_eq_shape(int rows, int hq, int hd, int dtype, long long part_rows,
                                        int cus) {
  AttnEqShape e{0, 0, 0, false};
  if (dtype != AKVS_BF16 || rows <= 0 || hq <= 0 || (hd != 64 && hd != 128)) return e;
  const int p128 = 2 * cus / hq, p256 = cus / hq;
  const int nt128 = (rows + 127) / 128, nt256 = (rows + 255) / 256;
  if (nt128 >= 3 && 4 * nt128 <= 3 * p128) {
    e.rb = 128;
    e.budget = p128;
  } else if (p256 >= 1 && 2 * nt256 <= p256) {
    e.rb = 256;
    e.budget = p256;
  } else if (p256 >= 1 && nt256 < 2 * p256) {
    e.rb = 256;
    e.budget = 2 * p256;
  } else {
    return e;
  }
  if ((rows + e.rb - 1) / e.rb > 64) return e;
  e.max_pc = (int)std::min<long long>(kAttnMaxPieces, part_rows / rows);
  e.use = e.max_pc >= 2;
  return e;
}

// The plan (one wave): tile t of rb rows sees kt_t = ceil(keys_t / 64) key tiles, keys_t
// its last row's position + 1. It is cut into c_t = ceil(kt_t / L) ranges of nearly equal
// length, L the smallest with sum_t c_t <= max(tiles, budget) and c_t <= max_pc. Items
// (tile, range) are numbered by the tile's range length, longest first (equal lengths:
// later tile first), a tile's ranges together. plan[0] = {tiles, items, max_t c_t},
// plan[1 + t] = {c_t, first item of tile t, kt_t} (c_t = 0 past the last tile).
__global__ __launch_bounds__(64) void k_attn_plan(const int32_t *pos, int pos0, int rows,
                                                  const int32_t *rows_dev,
                                                  const int32_t *row_base, int n_keys, int rb,
                                                  int budget, int max_pc, int4 *plan) {
  const int lane = threadIdx.x;
  int R = rows;
  if (rows_dev) R = min(R, *rows_dev);
  if (row_base && pos) pos += *row_base;
  const int nt = (R + rb - 1) / rb;
  int kt = 0;
  if (lane < nt) {
    const int e = min((lane + 1) * rb, R) - 1;
    kt = (min(n_keys, (pos ? pos[e] : pos0 + e) + 1) + 63) >> 6;
  }
  int ktmax = kt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) ktmax = max(ktmax, __shfl_xor(ktmax, o, 64));
  const int B = max(nt, budget);
  int lo = max(1, (ktmax + max_pc - 1) / max_pc), hi = max(lo, ktmax);
  while (lo < hi) {  // the same bounds in every lane
    const int L = (lo + hi) >> 1;
    int c = lane < nt ? (kt + L - 1) / L : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) c += __shfl_xor(c, o, 64);
    if (c <= B) hi = L;
    else lo = L + 1;
  }
  const int c = lane < nt ? (kt + lo - 1) / lo : 0;
  const int p = lane < nt ? (kt + c - 1) / c : 0;  // the tile's longest range
  int off = 0, total = 0, cmax = 0;
  for (int u = 0; u < nt; ++u) {  // u is the same in every lane: lane reads, no LDS trips
    const int pu = __builtin_amdgcn_readlane(p, u), cu = __builtin_amdgcn_readlane(c, u);
    if (pu > p || (pu == p && u > lane)) off += cu;
    total += cu;
    cmax = max(cmax, cu);
  }
  plan[1 + lane] = make_int4(c, off, kt, 0);
  if (lane == 0) plan[0] = make_int4(nt, total, cmax, 0);
}

// A block serves head group hg of KV head kvh: 32 * nrb query rows x gh query heads. Wave
// w owns 32 rows (row block w / gh) of query head kvh * G + hg * gh + w % gh. Waves 0-3
// stage each 64-key K / V tile in LDS for all of them (double buffered, the next tile in
// flight during the current one: hd 128 straight from global memory into LDS, hd 64 through
// registers). Block b serves KV head b % Hkv, so the blocks streaming one head's keys run on
// the same XCD and share its L2.
template <int HD, bool PREF>
__global__ __launch_bounds__(512) void k_attn_bf16(const bf16_t *__restrict__ Q,
                                                   const int32_t *pos, int pos0, int rows,
                                                   const int32_t *rows_dev,
                                                   const bf16_t *__restrict__ Kc,
                                                   const bf16_t *__restrict__ Vc, int n_keys,
                                                   int hq, int hkv, int gh, int n_groups,
                                                   int nrb, int n_tiles, int n_splits,
                                                   int split_keys,
                                                   float scale_log2,
                                                   bf16_t *__restrict__ out,
                                                   bf16_t *__restrict__ part_o,
                                                   float *__restrict__ part_ml,
                                                   const int32_t *row_base,
                                                   const int4 *__restrict__ plan) {
  constexpr int KS = HD / 16;          // contraction steps of S
  constexpr int DB = HD / 32;          // 32-wide head-dim blocks of O
  constexpr int KST = HD + 8;          // K tile row stride (bf16)
  constexpr int VRS = HD + 32;         // V tile row stride (bf16)
  constexpr int CPK = HD / 8;          // 16-byte chunks per key row
  constexpr int LT = 256;              // loading threads (waves 0-3)
  constexpr int KCH = 64 * CPK / LT;   // K (and V) chunks per loading thread
  // DIR: the tiles go from global memory straight into LDS (hd 128; PREF: hd 64, 4 waves)
  constexpr bool DIR = !PREF && HD == 128;
  constexpr int KBUF = DIR ? 64 * HD : 64 * KST, VBUF = DIR ? 64 * HD : 64 * VRS;
  // the two buffers of a tile pair; with DIR separate LDS objects (see the loop below)
  __shared__ __attribute__((aligned(16))) bf16_t Ks[(DIR ? 1 : 2) * KBUF];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[(DIR ? 1 : 2) * VBUF];
  __shared__ __attribute__((aligned(16))) bf16_t Ks1[DIR ? KBUF : 1];
  __shared__ __attribute__((aligned(16))) bf16_t Vt1[DIR ? VBUF : 1];
  __shared__ int s_max[8];
  if (row_base) {  // this call's rows start at row *row_base of q, pos and out
    const int rb0 = *row_base;
    Q += (size_t)rb0 * hq * HD;
    out += (size_t)rb0 * hq * HD;
    if (pos) pos += rb0;
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nw = blockDim.x >> 6;
  const bool loader = wave < 4;
  const int G = hq / hkv;
  const int kvh = blockIdx.x % hkv;
  int rest = (int)(blockIdx.x / hkv);
  const int hg = rest % n_groups;
  rest /= n_groups;
  const int head = kvh * G + hg * gh + wave % gh;
  int R = rows;
  if (rows_dev) R = min(R, *rows_dev);
  const int rb_rows = 32 * nrb;
  int split, tile, n_part = n_splits, kv_begin = -1;
  if (plan) {  // item `rest` of the call's plan (see k_attn_plan)
    const int4 e = plan[1 + lane];  // (c = 0 past the last tile)
    const unsigned long long mine = __ballot(e.x > 0 && e.y <= rest && rest < e.y + e.x);
    if (mine == 0) return;  // past the last item (the whole block)
    const int t = __ffsll((long long)mine) - 1;
    const int c = __shfl(e.x, t, 64), first = __shfl(e.y, t, 64), kt = __shfl(e.z, t, 64);
    tile = t;
    split = rest - first;
    n_part = c;
    if (c > n_splits) return;  // not a plan for this launch's partial slots
    kv_begin = (split * kt / c) * 64;
    split_keys = ((split + 1) * kt / c) * 64 - kv_begin;
  } else {
    split = rest % n_splits;
    tile = n_tiles - 1 - rest / n_splits;
  }
  const int row0 = tile * rb_rows;
  if (tile < 0 || row0 >= R) return;
  const int hi = lane >> 5;  // which half of a row's 32 keys (and 32 dims) this lane holds
  const int r = row0 + (wave / gh) * 32 + (lane & 31);
  const bool rvalid = r < R;
  const int rp = rvalid ? (pos ? pos[r] : pos0 + r) : -1;
  const int rpos = rvalid ? rp : 0;
  int wmax = rp, wmin = rvalid ? rp : 0x7fffffff;
#pragma unroll
  for (int o = 1; o < 32; o <<= 1) {
    wmax = max(wmax, __shfl_xor(wmax, o, 64));
    wmin = min(wmin, __shfl_xor(wmin, o, 64));
  }
  if (lane == 0) s_max[wave] = wmax;
  __syncthreads();
  int bmax = -1;
  for (int w = 0; w < nw; ++w) bmax = max(bmax, s_max[w]);
  // this block's keys: [kv_begin, kv_end) of split `split`
  if (kv_begin < 0) kv_begin = split * split_keys;
  const int kv_end = min(min(n_keys, bmax + 1), kv_begin + split_keys);
  const int nkt = kv_end > kv_begin ? (kv_end - kv_begin + 63) / 64 : 0;
  const size_t prow = ((size_t)split * rows + r) * hq + head;  // partial slot of this lane's row
  if (nkt == 0) {
    if (n_splits > 1 && rvalid && hi == 0) {
      part_ml[2 * prow] = -INFINITY;
      part_ml[2 * prow + 1] = 0.f;
    }
    return;
  }

  // Q^T operand of S: lane holds dims ks*16 + hi*8 .. +7 of its row
  bf16x8_t qf[KS];
  {
    const bf16_t *qrow = Q + ((size_t)(rvalid ? r : row0) * hq + head) * HD + hi * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8_t *>(qrow + ks * 16);
    // vmcnt(0): the query fragments are complete before the key loop, so the loop's waits
    // on the K / V prefetch never cover them
    __builtin_amdgcn_s_waitcnt(0x0f70);
  }
  f32x16_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;  // l_run: this lane's half of the row sum

  // One K / V tile in the loading waves' registers. Keys past kv_end are clamped to the
  // last key: finite data that the score mask gives probability 0.
  u32x4_t kreg[DIR ? 1 : KCH], vreg[DIR ? 1 : KCH];
  const int klast = kv_end - 1;
  // DIR staging: global_load_lds, 16 bytes per lane, the 64 lanes of a loading wave filling
  // 1 KB = 4 unpadded rows of 256 bytes (lane p: row +p/16, 16-byte chunk position p%16).
  // Which global chunk a lane fetches sets the layout: chunk c of row r sits at position
  // c ^ (r & 15) for K and c ^ 4 (r & 3) for V, so that the 32 K rows of a fragment read
  // and the 4 V rows of a transposing read fall on distinct banks. No registers, no LDS
  // stores in the loading waves: 4.7 % faster on the 32B probe layer (986 -> 940 us), same
  // bits. The transposing V reads are inline assembly: through the builtin, the compiler
  // cannot tell them from the DMA's LDS writes and waits for the next tile's DMA before the
  // first of them, which cost the 4-wave blocks 20-27 % against register staging with
  // read-ahead; without that wait the 4-wave blocks are 3-8 % faster than the register
  // staging on the 3B probe layers (1/100 to 3/10 of the context), the 8-wave blocks about
  // 1 % (standalone harness, not in the repository).
  auto dma_to = [&](int key0_, bf16_t *kbuf, bf16_t *vbuf) {
    const int w = tid >> 6;  // loading wave 0..3
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (i * 4 + w) * 4 + (lane >> 4);
      const int pc = lane & 15;
      const size_t gro = ((size_t)min(key0_ + row, klast) * hkv + kvh) * HD;
      __builtin_amdgcn_global_load_lds((const void *)(Kc + gro + (pc ^ (row & 15)) * 8),
                                       (__attribute__((address_space(3))) void *)(
                                           kbuf + (i * 4 + w) * 4 * HD),
                                       16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void *)(Vc + gro + (pc ^ (4 * (row & 3))) * 8),
                                       (__attribute__((address_space(3))) void *)(
                                           vbuf + (i * 4 + w) * 4 * HD),
                                       16, 0, 0);
    }
  };
#define AKVS_KV_LOAD(KEY0)                                                                  \
  {                                                                                         \
    _Pragma("unroll") for (int i = 0; i < KCH; ++i) {                                       \
      const int c = tid + LT * i, kr = c / CPK, e0 = (c - kr * CPK) * 8;                    \
      const size_t o_ = ((size_t)min((KEY0) + kr, klast) * hkv + kvh) * HD + e0;            \
      kreg[i] = *reinterpret_cast<const u32x4_t *>(Kc + o_);                                \
      vreg[i] = *reinterpret_cast<const u32x4_t *>(Vc + o_);                                \
    }                                                                                       \
  }
#define AKVS_KV_STORE(KB, VB)                                                               \
  {                                                                                         \
    bf16_t *ks_ = (KB);                                                                     \
    bf16_t *vt_ = (VB);                                                                     \
    _Pragma("unroll") for (int i = 0; i < KCH; ++i) {                                       \
      const int c = tid + LT * i, kr = c / CPK, e0 = (c - kr * CPK) * 8;                    \
      *reinterpret_cast<u32x4_t *>(ks_ + kr * KST + e0) = kreg[i];                          \
      *reinterpret_cast<u32x4_t *>(vt_ + kr * VRS + e0) = vreg[i];                          \
    }                                                                                       \
  }

  if (DIR) {
    if (loader) dma_to(kv_begin, Ks, Vt);
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  } else if (loader) {
    AKVS_KV_LOAD(kv_begin);
    AKVS_KV_STORE(Ks, Vt);
  }
  __syncthreads();
  // one 64-key tile from ks_ / vt_, the next one staged into nks_ / nvt_
  auto step = [&](int kt, const bf16_t *ks_in, const bf16_t *vt_in, bf16_t *nks_,
                  bf16_t *nvt_) __attribute__((always_inline)) {
    const bf16_t *ks_ = DIR ? ks_in : Ks + (kt & 1) * KBUF;
    const bf16_t *vt_ = DIR ? vt_in : Vt + (kt & 1) * VBUF;
    const int key0 = kv_begin + kt * 64;
    const bool more = kt + 1 < nkt;
    if (loader && more) {
      if (DIR) dma_to(key0 + 64, nks_, nvt_);
      else AKVS_KV_LOAD(key0 + 64);
    }
    // PREF (register-staged hd 64 blocks): the K fragments of a 32-key block are read ahead
    // (the tile's first block here, its second under the first block's softmax) and each
    // block's V^T fragments are requested before its score MFMAs, so no MFMA waits on its own
    // LDS read. It needs about 50 more registers.
    bf16x8_t kf[KS];
    if (PREF && key0 <= wmax) {
      const bf16_t *krow = ks_ + (lane & 31) * KST + hi * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kf[ks] = *reinterpret_cast<const bf16x8_t *>(krow + ks * 16);
      static_assert(!DIR || !PREF, "the read-ahead reads the padded K layout");
    }
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int sk0 = key0 + st * 32;
      if (sk0 <= wmax) {  // skip keys past every row of this wave
        // V^T operand of k-step t, head-dim block db: lane holds dim db*32 + lane%32 at the
        // keys of its 8 slots (slots 0-3: 16t + 4*hi + 0..3 of this 32-key block, 4-7: the
        // same + 8), two transposing reads of 4 keys each
        bf16x8_t vf[2][DB];
        auto read_v = [&](int t, int db) {
          typedef short v4s __attribute__((ext_vector_type(4)));
          // DIR: the 16-byte chunk db*4 + 2*((lane>>4)&1) + (lane&3)/2 of a row whose low two
          // bits are (lane>>2)&3 sits at db ^ ((lane>>2)&3) in place of db
          const bf16_t *vb =
              DIR ? vt_ + (st * 32 + 16 * t + 4 * hi + ((lane & 15) >> 2)) * HD +
                        (4 * (db ^ ((lane >> 2) & 3)) + 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) * 8 +
                        (lane & 1) * 4
                  : vt_ + (st * 32 + 16 * t + 4 * hi + ((lane & 15) >> 2)) * VRS + db * 32 +
                        16 * ((lane >> 4) & 1) + 4 * (lane & 3);
          uint32_t vw[4];
          if constexpr (DIR) {
            // as assembly: the builtin carries no alias information, so the compiler would
            // wait for the next tile's DMA (vmcnt(0)) before it; the fragments are complete
            // at the explicit lgkmcnt(0) before the P.V MFMAs (below)
            typedef unsigned int u2_t __attribute__((ext_vector_type(2)));
            u2_t x0, x1;
            const uint32_t a0 =
                (uint32_t)(size_t)(__attribute__((address_space(3))) const bf16_t *)(vb);
            asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(x0) : "v"(a0));
            asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(x1) : "v"(a0), "i"(8 * HD * 2));
            vw[0] = x0.x; vw[1] = x0.y; vw[2] = x1.x; vw[3] = x1.y;
          } else {
            const v4s r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) v4s *)(vb));
            const v4s r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) v4s *)(vb + 8 * VRS));
            uint2 x0, x1;
            __builtin_memcpy(&x0, &r0, 8);
            __builtin_memcpy(&x1, &r1, 8);
            vw[0] = x0.x; vw[1] = x0.y; vw[2] = x1.x; vw[3] = x1.y;
          }
          __builtin_memcpy(&vf[t][db], vw, 16);
        };
        if (PREF || DIR) {  // every V^T fragment of the block requested up front
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int db = 0; db < DB; ++db) read_v(t, db);
        }
        // S^T block: 32 keys x 32 rows; s[i] is key sk0 + (i/4)*8 + hi*4 + i%4 of row r
        f32x16_t sc;
#pragma unroll
        for (int i = 0; i < 16; ++i) sc[i] = 0.f;
        // K fragment of step ks: 16-byte chunk 2ks + hi of row st*32 + lane%32 (DIR: at its
        // swizzled position; st*32 is a multiple of 16, so the row's low bits are lane%16)
        const bf16_t *krow =
            ks_ + (st * 32 + (lane & 31)) * (DIR ? HD : KST) + (DIR ? 0 : hi * 8);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8_t a =
              PREF ? kf[ks]
                   : *reinterpret_cast<const bf16x8_t *>(
                         krow + (DIR ? ((2 * ks + hi) ^ (lane & 15)) * 8 : ks * 16));
          sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sc, 0, 0, 0);
        }
        if (PREF && st == 0 && sk0 + 32 <= wmax) {
          const bf16_t *knext = ks_ + (32 + (lane & 31)) * KST + hi * 8;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            kf[ks] = *reinterpret_cast<const bf16x8_t *>(knext + ks * 16);
        }
        if (sk0 + 31 > wmin || sk0 + 31 >= kv_end) {  // causal / range mask needed
          // score i is key sk0 + hi*4 + (i/4)*8 + i%4: masked past min(row position, last key)
          const int lim = min(rpos, kv_end - 1) - (sk0 + hi * 4);
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if ((i >> 2) * 8 + (i & 3) > lim) sc[i] = -INFINITY;
        }
        float mx = sc[0];
#pragma unroll
        for (int i = 1; i < 16; ++i) mx = fmaxf(mx, sc[i]);
        // raise the running maximum only when some score exceeds it by more than 2^8
        if (__ballot(mx * scale_log2 > m_run + 8.f)) {
          const float mp = fmaxf(mx, __shfl_xor(mx, 32, 64)) * scale_log2;
          const float m_new = fmaxf(m_run, mp);
          const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
          for (int db = 0; db < DB; ++db) o[db] *= alpha;
          l_run *= alpha;
          m_run = m_new;
        }
        // rows with no key yet keep m = -inf: offset by 0 then (every p is 0)
        const float m_off = m_run == -INFINITY ? 0.f : m_run;
        float pv[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          pv[i] = __builtin_amdgcn_exp2f(fmaf(sc[i], scale_log2, -m_off));  // v_exp_f32: arguments <= 8
          l_run += pv[i];
        }
        if constexpr (DIR) {  // the assembly reads above: results complete here
          static_assert(DB == 4, "hd 128");
          asm volatile("s_waitcnt lgkmcnt(0)"
                       : "+v"(vf[0][0]), "+v"(vf[0][1]), "+v"(vf[0][2]), "+v"(vf[0][3]),
                         "+v"(vf[1][0]), "+v"(vf[1][1]), "+v"(vf[1][2]), "+v"(vf[1][3]));
        }
        // P^T operand of k-step t: slots hi*8 + j hold keys 16t + (j/4)*8 + hi*4 + j%4
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          uint32_t pw[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) pw[j] = pack_bf2(pv[8 * t + 2 * j], pv[8 * t + 2 * j + 1]);
          bf16x8_t pb;
          __builtin_memcpy(&pb, pw, 16);
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            if (!PREF && !DIR) read_v(t, db);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[t][db], pb, o[db], 0, 0, 0);
          }
        }
      }
    }
    if (DIR) __builtin_amdgcn_s_waitcnt(0x0f70);  // this wave's DMA of the next tile landed
    else if (loader && more) AKVS_KV_STORE(Ks + ((kt + 1) & 1) * KBUF, Vt + ((kt + 1) & 1) * VBUF);
    __syncthreads();
  };
  if constexpr (DIR) {
    // unrolled by two over separate LDS objects, so that the compiler can see that a
    // step's reads and the next tile's DMA touch different memory and does not wait for
    // the DMA before the reads
    for (int kt = 0; kt < nkt; kt += 2) {
      step(kt, Ks, Vt, Ks1, Vt1);
      if (kt + 1 < nkt) step(kt + 1, Ks1, Vt1, Ks, Vt);
    }
  } else {
    // (the same step written out in the loop: as a lambda it cost the read-ahead variant
    // two spilled registers)
    for (int kt = 0; kt < nkt; ++kt) {
    const bf16_t *ks_ = Ks + (kt & 1) * KBUF;
    const bf16_t *vt_ = Vt + (kt & 1) * VBUF;
    const int key0 = kv_begin + kt * 64;
    const bool more = kt + 1 < nkt;
    if (loader && more) {
      AKVS_KV_LOAD(key0 + 64);
    }
    // PREF (register-staged hd 64 blocks): the K fragments of a 32-key block are read ahead
    // (the tile's first block here, its second under the first block's softmax) and each
    // block's V^T fragments are requested before its score MFMAs, so no MFMA waits on its own
    // LDS read. It needs about 50 more registers.
    bf16x8_t kf[KS];
    if (PREF && key0 <= wmax) {
      const bf16_t *krow = ks_ + (lane & 31) * KST + hi * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kf[ks] = *reinterpret_cast<const bf16x8_t *>(krow + ks * 16);
      static_assert(!DIR || !PREF, "the read-ahead reads the padded K layout");
    }
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int sk0 = key0 + st * 32;
      if (sk0 <= wmax) {  // skip keys past every row of this wave
        // V^T operand of k-step t, head-dim block db: lane holds dim db*32 + lane%32 at the
        // keys of its 8 slots (slots 0-3: 16t + 4*hi + 0..3 of this 32-key block, 4-7: the
        // same + 8), two transposing reads of 4 keys each
        bf16x8_t vf[2][DB];
        auto read_v = [&](int t, int db) {
          typedef short v4s __attribute__((ext_vector_type(4)));
          // DIR: the 16-byte chunk db*4 + 2*((lane>>4)&1) + (lane&3)/2 of a row whose low two
          // bits are (lane>>2)&3 sits at db ^ ((lane>>2)&3) in place of db
          const bf16_t *vb =
              DIR ? vt_ + (st * 32 + 16 * t + 4 * hi + ((lane & 15) >> 2)) * HD +
                        (4 * (db ^ ((lane >> 2) & 3)) + 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) * 8 +
                        (lane & 1) * 4
                  : vt_ + (st * 32 + 16 * t + 4 * hi + ((lane & 15) >> 2)) * VRS + db * 32 +
                        16 * ((lane >> 4) & 1) + 4 * (lane & 3);
          const v4s r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) v4s *)(vb));
          const v4s r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) v4s *)(vb + 8 * (DIR ? HD : VRS)));
          uint2 x0, x1;
          __builtin_memcpy(&x0, &r0, 8);
          __builtin_memcpy(&x1, &r1, 8);
          uint32_t vw[4] = {x0.x, x0.y, x1.x, x1.y};
          __builtin_memcpy(&vf[t][db], vw, 16);
        };
        if (PREF) {
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int db = 0; db < DB; ++db) read_v(t, db);
        }
        // S^T block: 32 keys x 32 rows; s[i] is key sk0 + (i/4)*8 + hi*4 + i%4 of row r
        f32x16_t sc;
#pragma unroll
        for (int i = 0; i < 16; ++i) sc[i] = 0.f;
        // K fragment of step ks: 16-byte chunk 2ks + hi of row st*32 + lane%32 (DIR: at its
        // swizzled position; st*32 is a multiple of 16, so the row's low bits are lane%16)
        const bf16_t *krow =
            ks_ + (st * 32 + (lane & 31)) * (DIR ? HD : KST) + (DIR ? 0 : hi * 8);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8_t a =
              PREF ? kf[ks]
                   : *reinterpret_cast<const bf16x8_t *>(
                         krow + (DIR ? ((2 * ks + hi) ^ (lane & 15)) * 8 : ks * 16));
          sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sc, 0, 0, 0);
        }
        if (PREF && st == 0 && sk0 + 32 <= wmax) {
          const bf16_t *knext = ks_ + (32 + (lane & 31)) * KST + hi * 8;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            kf[ks] = *reinterpret_cast<const bf16x8_t *>(knext + ks * 16);
        }
        if (sk0 + 31 > wmin || sk0 + 31 >= kv_end) {  // causal / range mask needed
          // score i is key sk0 + hi*4 + (i/4)*8 + i%4: masked past min(row position, last key)
          const int lim = min(rpos, kv_end - 1) - (sk0 + hi * 4);
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if ((i >> 2) * 8 + (i & 3) > lim) sc[i] = -INFINITY;
        }
        float mx = sc[0];
#pragma unroll
        for (int i = 1; i < 16; ++i) mx = fmaxf(mx, sc[i]);
        // raise the running maximum only when some score exceeds it by more than 2^8
        if (__ballot(mx * scale_log2 > m_run + 8.f)) {
          const float mp = fmaxf(mx, __shfl_xor(mx, 32, 64)) * scale_log2;
          const float m_new = fmaxf(m_run, mp);
          const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
          for (int db = 0; db < DB; ++db) o[db] *= alpha;
          l_run *= alpha;
          m_run = m_new;
        }
        // rows with no key yet keep m = -inf: offset by 0 then (every p is 0)
        const float m_off = m_run == -INFINITY ? 0.f : m_run;
        float pv[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          pv[i] = __builtin_amdgcn_exp2f(fmaf(sc[i], scale_log2, -m_off));  // v_exp_f32: arguments <= 8
          l_run += pv[i];
        }
        // P^T operand of k-step t: slots hi*8 + j hold keys 16t + (j/4)*8 + hi*4 + j%4
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          uint32_t pw[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) pw[j] = pack_bf2(pv[8 * t + 2 * j], pv[8 * t + 2 * j + 1]);
          bf16x8_t pb;
          __builtin_memcpy(&pb, pw, 16);
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            if (!PREF) read_v(t, db);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[t][db], pb, o[db], 0, 0, 0);
          }
        }
      }
    }
    if (loader && more) AKVS_KV_STORE(Ks + ((kt + 1) & 1) * KBUF, Vt + ((kt + 1) & 1) * VBUF);
    __syncthreads();
    }
  }
#undef AKVS_KV_LOAD
#undef AKVS_KV_STORE
  const float l_row = l_run + __shfl_xor(l_run, 32, 64);
  if (!rvalid) return;
  // o[db][i] is dim db*32 + (i/4)*8 + hi*4 + i%4 of row r
  if (n_splits > 1 && n_part == 1) {  // a whole tile: final output here; the merge skips
    if (hi == 0) {                     // the row (end mark in the first slot)
      part_ml[2 * prow] = -INFINITY;
      part_ml[2 * prow + 1] = -1.f;
    }
  } else if (n_splits > 1) {  // this split's output over its own keys (bf16) + (max, sum)
    const float pinv = l_row > 0.f ? 1.0f / l_row : 0.f;  // no visible key: m = -inf, skipped
    bf16_t *po = part_o + prow * HD + hi * 4;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        store4(po + db * 32 + q4 * 8, o[db][4 * q4] * pinv, o[db][4 * q4 + 1] * pinv,
               o[db][4 * q4 + 2] * pinv, o[db][4 * q4 + 3] * pinv);
    if (hi == 0) {
      part_ml[2 * prow] = m_run;
      part_ml[2 * prow + 1] = l_row;
      if (split == n_part - 1 && n_part < n_splits) {  // end mark: no later split of this tile
        const size_t pend = ((size_t)n_part * rows + r) * hq + head;
        part_ml[2 * pend] = -INFINITY;
        part_ml[2 * pend + 1] = -1.f;
      }
    }
    return;
  }
  const float inv = 1.0f / l_row;
  bf16_t *orow = out + ((size_t)r * hq + head) * HD + hi * 4;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4)
      store4(orow + db * 32 + q4 * 8, o[db][4 * q4] * inv, o[db][4 * q4 + 1] * inv,
             o[db][4 * q4 + 2] * inv, o[db][4 * q4 + 3] * inv);
}

// Merge of the key splits of one (row, head): split s holds its output over its own keys,
// o_s (bf16, normalised by its own sum l_s), and (m_s, l_s); the result is
// sum_s w_s o_s / sum_s w_s with w_s = 2^(m_s - max m) l_s, added in split order. A split
// whose keys all lie past the row (causal mask) holds m = -inf and is skipped, never
// multiplied in (its part_o slot holds whatever the workspace held). With a device-planned
// split a tile may use fewer splits than the launch's count: l = -1 after its last one
// ends the list (the slots past it are stale); l = -1 in the first slot marks a row whose
// tile ran as one piece and whose output the attention block wrote itself.
// Thread = 8 consecutive head dims of one (row, head) (16-byte loads and stores). Up to 8
// splits, all (m, l) pairs and partial outputs are requested at once; with more, the
// maxima first, then the splits in order.
__global__ __launch_bounds__(256) void k_attn_combine(const bf16_t *__restrict__ part_o,
                                                      const float *__restrict__ part_ml,
                                                      int n_splits, int rows,
                                                      const int32_t *rows_dev, int hq, int hd,
                                                      bf16_t *__restrict__ out,
                                                      const int32_t *row_base,
                                                      const int4 *plan) {
  const int per = hd >> 3;  // threads per (row, head)
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long item = gid / per;
  const int e0 = (int)(gid - item * per) * 8;
  int R = rows;
  if (rows_dev) R = min(R, *rows_dev);
  if (item >= (long long)R * hq) return;
  if (row_base) out += (size_t)*row_base * hq * hd;
  if (plan) n_splits = min(n_splits, plan[0].z);  // no tile of the plan has more pieces
  const size_t stride = (size_t)rows * hq;  // items per split
  float mx = -INFINITY, l = 0.f, a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = 0.f;
  if (n_splits <= 8) {  // every partial of this item requested at once
    float2 ml[8];
    float o[8][8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (u < n_splits) {
        const size_t pi = u * stride + item;
        ml[u] = *reinterpret_cast<const float2 *>(part_ml + 2 * pi);
        load8(part_o + pi * hd + e0, o[u]);
      }
    }
    int n = n_splits;  // up to the first end mark
#pragma unroll
    for (int u = 7; u >= 0; --u)
      if (u < n_splits && ml[u].y < 0.f) n = u;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (u < n) mx = fmaxf(mx, ml[u].x);
    if (n == 0) return;  // the attention wrote this row's output itself
    const float moff = mx == -INFINITY ? 0.f : mx;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (u >= n || ml[u].x == -INFINITY) continue;
      const float w = exp2f(ml[u].x - moff) * ml[u].y;
      l += w;
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] += w * o[u][i];
    }
  } else {
    int n = n_splits;  // up to the first end mark
    for (int sp = 0; sp < n; ++sp) {
      const float2 ml = *reinterpret_cast<const float2 *>(part_ml + 2 * (sp * stride + item));
      if (ml.y < 0.f) n = sp;
      else mx = fmaxf(mx, ml.x);
    }
    if (n == 0) return;
    const float moff = mx == -INFINITY ? 0.f : mx;
    for (int sp = 0; sp < n; ++sp) {
      const size_t pi = sp * stride + item;
      const float2 ml = *reinterpret_cast<const float2 *>(part_ml + 2 * pi);
      if (ml.x == -INFINITY) continue;  // no visible key: its part_o was never written
      float o[8];
      load8(part_o + pi * hd + e0, o);
      const float w = exp2f(ml.x - moff) * ml.y;
      l += w;
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] += w * o[i];
    }
  }
  const float inv = 1.0f / l;
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] *= inv;
  store8(out + item * hd + e0, a);
}

// fp32 path (small models): one wave per (row, head), keys in tiles of 64, online softmax.
template <int HD>
__global__ __launch_bounds__(64) void k_attn_f32(const float *__restrict__ Q, const int32_t *pos,
                                                 int pos0, int rows, const int32_t *rows_dev,
                                                 const float *__restrict__ Kc,
                                                 const float *__restrict__ Vc, int n_keys, int hq,
                                                 int hkv, float scale, float *__restrict__ out,
                                                 const int32_t *row_base) {
  constexpr int PER = HD / 64;
  __shared__ float qs[HD];
  __shared__ float ps[64];
  const int lane = threadIdx.x;
  const int r = blockIdx.x, head = blockIdx.y;
  if (row_base) {
    const int rb0 = *row_base;
    Q += (size_t)rb0 * hq * HD;
    out += (size_t)rb0 * hq * HD;
    if (pos) pos += rb0;
  }
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
  const AttnShape a = attn_shape(hq / hkv, rows, hkv);
  if (a.gh == 0 || rows <= 0) return 1;
  const int rb = 32 * a.nrb;
  const long long base = (long long)((rows + rb - 1) / rb) * hkv * a.n_groups;
  if (base >= 512) return 1;                        // two blocks per compute unit already
  long long sp = (768 + base - 1) / base;           // else aim at ~768 blocks (measured)
  const long long cap = (n_keys + 255) / 256;        // at least 256 keys per split
  if (sp > cap) sp = cap;
  if (sp > 64) sp = 64;
  return sp < 1 ? 1 : (int)sp;
}

int attn_split_keys(int n_keys, int n_splits) {
  const int per = (n_keys + n_splits - 1) / n_splits;
  return (per + 63) / 64 * 64;
}

int attn_part_splits(int rows, int hq, int hkv, int hd, int n_keys) {
  const int sp = attn_splits(rows, hq, hkv, n_keys);
  const AttnEqShape e =
      attn_eq_shape(rows, hq, hd, AKVS_BF16, (long long)kAttnMaxPieces * rows, gemm_cu_count());
  return e.use ? std::max(sp, kAttnMaxPieces) : sp;
}

hipError_t launch_attention_plan(const int32_t *pos, int pos0, int rows, const int32_t *rows_dev,
                                 int n_keys, int hq, int hd, int dtype, long long part_rows,
                                 int32_t *plan, hipStream_t s, const int32_t *row_base) {
  const AttnEqShape e = attn_eq_shape(rows, hq, hd, dtype, part_rows, gemm_cu_count());
  if (!e.use || !plan) return hipSuccess;  // launch_attention will not read it either
  hipLaunchKernelGGL(k_attn_plan, dim3(1), dim3(64), 0, s, pos, pos0, rows, rows_dev, row_base,
                     n_keys, e.rb, e.budget, e.max_pc, reinterpret_cast<int4 *>(plan));
  return hipGetLastError();
}

hipError_t launch_attention(const void *q, const int32_t *pos, int pos0, int rows,
                            const int32_t *rows_dev, const void *k, const void *v, int n_keys,
                            int hq, int hkv, int hd, int dtype, void *out, float *part_o,
                            float *part_ml, long long part_rows, hipStream_t s,
                            const int32_t *row_base, const int32_t *plan) {
  if (rows == 0) return hipSuccess;
  if (dtype == AKVS_BF16) {
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    const bf16_t *Q = reinterpret_cast<const bf16_t *>(q);
    const bf16_t *K = reinterpret_cast<const bf16_t *>(k);
    const bf16_t *V = reinterpret_cast<const bf16_t *>(v);
    bf16_t *O = reinterpret_cast<bf16_t *>(out);
    AttnShape a = attn_shape(hq / hkv, rows, hkv);
    if (a.gh == 0) return hipErrorInvalidValue;
    const AttnEqShape e = attn_eq_shape(rows, hq, hd, dtype, part_rows, gemm_cu_count());
    if (plan && part_o && part_ml && e.use) {  // the split that launch_attention_plan planned
      const int nrb = e.rb / 32;
      const int items = std::max((rows + e.rb - 1) / e.rb, e.budget);
      dim3 g(items * hq), b(64 * nrb);
      const int4 *P = reinterpret_cast<const int4 *>(plan);
#define AKVS_ATTN_PLANNED(HD_, PREF_)                                                             \
  hipLaunchKernelGGL((k_attn_bf16<HD_, PREF_>), g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V,     \
                     n_keys, hq, hkv, 1, hq / hkv, nrb, 1, e.max_pc, 0, scale_log2, O,             \
                     reinterpret_cast<bf16_t *>(part_o), part_ml, row_base, P)
      if (hd == 128) {
        AKVS_ATTN_PLANNED(128, false);
      } else {
        if (nrb == 4) AKVS_ATTN_PLANNED(64, true); else AKVS_ATTN_PLANNED(64, false);
      }
#undef AKVS_ATTN_PLANNED
      hipError_t er = hipGetLastError();
      if (er != hipSuccess) return er;
      const long long threads = (long long)rows * hq * (hd / 8);
      hipLaunchKernelGGL(k_attn_combine, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                         reinterpret_cast<const bf16_t *>(part_o), part_ml, e.max_pc, rows,
                         rows_dev, hq, hd, O, row_base, P);
      return hipGetLastError();
    }
    int n_splits = part_o && part_ml ? attn_splits(rows, hq, hkv, n_keys) : 1;
    if ((long long)n_splits * rows > part_rows) n_splits = (int)std::max(1LL, part_rows / rows);
    const int split_keys = attn_split_keys(n_keys, n_splits);
    const int n_tiles = (rows + 32 * a.nrb - 1) / (32 * a.nrb);
    dim3 g(n_tiles * hkv * a.n_groups * n_splits), b(64 * a.nrb * a.gh);
    const bool pref = a.nrb * a.gh <= 4;  // hd 64 (see PREF in the kernel)
#define AKVS_ATTN(HD_, PREF_)                                                                    \
  hipLaunchKernelGGL((k_attn_bf16<HD_, PREF_>), g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V,    \
                     n_keys, hq, hkv, a.gh, a.n_groups, a.nrb, n_tiles, n_splits, split_keys,      \
                     scale_log2, O, reinterpret_cast<bf16_t *>(part_o), part_ml, row_base,         \
                     nullptr)
    if (hd == 128) {
      AKVS_ATTN(128, false);  // the direct-to-LDS staging, 4- and 8-wave blocks alike
    } else {
      if (pref) AKVS_ATTN(64, true); else AKVS_ATTN(64, false);
    }
#undef AKVS_ATTN
    if (n_splits > 1) {
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      const long long threads = (long long)rows * hq * (hd / 8);
      hipLaunchKernelGGL(k_attn_combine, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                         reinterpret_cast<const bf16_t *>(part_o), part_ml, n_splits, rows,
                         rows_dev, hq, hd, O, row_base, nullptr);
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
                         hq, hkv, scale, O, row_base);
    else
      hipLaunchKernelGGL(k_attn_f32<64>, g, b, 0, s, Q, pos, pos0, rows, rows_dev, K, V, n_keys,
                         hq, hkv, scale, O, row_base);
  }
  return hipGetLastError();
}

}  // namespace akvs
