// Host-side launchers of the akvs kernels. All launch on the given stream, return the
// HIP status of the launch and assume the caller validated every size and pointer.
#pragma once
#include "common.h"

namespace akvs {

// ---- k_misc.hip ---------------------------------------------------------------------
// table row i holds position p0 + i.
hipError_t launch_rope_table(int p0, int n_pos, int head_dim, double theta, float *table,
                             hipStream_t s);
// h[t][:] = embed[tok[t]][:] (fp32), t < n; ids outside [0, vocab) give a zero row.
hipError_t launch_embed(const int32_t *tok, int n, const void *embed, int dtype, int vocab, int D,
                        float *h, hipStream_t s);
// out[i] = RMSNorm(h[src(i)]) * gain, i < rows (and < *rows_dev if given).
// src(i) = i + (base_dev ? *base_dev - rows : 0)  (base_dev selects the last `rows` rows).
hipError_t launch_rmsnorm(const float *h, int ldh, int rows, const int32_t *rows_dev,
                          const int32_t *base_dev, const void *gain, int gain_dtype, int D,
                          float eps, void *out, int out_dtype, int ldo, hipStream_t s);
// dst[base + i] = src[idx[i]], i < *n_dev (rows of D floats; base = *dst_base or 0);
// indices outside [0, n_src) give 0.
hipError_t launch_gather_rows(const float *src, int n_src, const int32_t *idx, int cap,
                              const int32_t *n_dev, int D, float *dst, hipStream_t s,
                              const int32_t *dst_base = nullptr);
// dst row i = src row (base + *n_dev - n + i), i < n: the last n of *n_dev rows that start
// at row base = *src_base (or 0).
hipError_t launch_copy_tail_rows(const void *src, size_t row_bytes, int n, const int32_t *n_dev,
                                 void *dst, hipStream_t s, const int32_t *src_base = nullptr);
// row_off[b] = n_rows[0] + ... + n_rows[b-1] for b = 0..B (a batch's row segments).
hipError_t launch_batch_layout(const int32_t *n_rows, int B, int32_t *row_off, hipStream_t s);
// dst[*dst_base + i] = src[i] for i < min(cap, *n_dev).
hipError_t launch_copy_ints_at(const int32_t *src, int cap, const int32_t *n_dev, int32_t *dst,
                               const int32_t *dst_base, hipStream_t s);
// dst[0] = src[0] on the device.
hipError_t launch_copy_int(const int32_t *src, int32_t *dst, hipStream_t s);
// per unit token t < T_c: tok_delta[t] = s_i, tok_chunk[t] = i.
hipError_t launch_token_setup(const int32_t *meta, int n_chunks, int32_t *tok_delta,
                              int32_t *tok_chunk, hipStream_t s);

// ---- k_reuse.hip --------------------------------------------------------------------
hipError_t launch_divergence(const void *k_fresh, const void *v_fresh, int fresh_dtype,
                             CacheLayer cache, int n_tokens, int hkv, int hd,
                             const int32_t *tok_delta, const float *rope, int rope_rows,
                             float *d_k, float *d_v, hipStream_t s);
hipError_t launch_select(const float *d_k, const float *d_v, const int32_t *meta, int n_chunks,
                         int t_ctx, int q, uint32_t flags, int32_t *probe_k, int32_t *probe_v,
                         float *w_k, float *w_v, uint8_t *tok_flags, int32_t *chunk_rows,
                         int32_t *rows, int32_t *n_rows, int32_t *fresh_row, hipStream_t s);
hipError_t launch_chunk_offset(const void *k_fresh, const void *v_fresh, int fresh_dtype,
                               const int32_t *fresh_row, CacheLayer cache, const int32_t *meta,
                               int n_chunks, const int32_t *probe_k, const int32_t *probe_v,
                               uint32_t flags, int hkv, int hd, const float *rope, int rope_rows,
                               float *mu_k, float *mu_v, hipStream_t s,
                               const int32_t *fresh_base = nullptr);
// Corrected (or, with mu == nullptr and tok_flags == nullptr, just re-rotated) cache rows.
// A token's unit and offset come from tok_chunk / tok_delta when given, else from a
// binary search of meta (n_chunks entries).
hipError_t launch_correction(CacheLayer cache, const float *mu_k, const float *mu_v,
                             const float *w_k, const float *w_v, const uint8_t *tok_flags,
                             const void *k_fresh, const void *v_fresh, const int32_t *fresh_row,
                             const int32_t *tok_chunk, const int32_t *tok_delta,
                             const int32_t *meta, int n_chunks, int t_ctx,
                             int t_all, int hkv, int hd, uint32_t flags, const float *rope,
                             int rope_rows, void *k_corr, void *v_corr, int out_dtype,
                             hipStream_t s,
                             const int32_t *fresh_base = nullptr);
hipError_t launch_quantize(const void *x, int x_dtype, int n_rows, int hd, int bits,
                           uint8_t *codes, _Float16 *meta, hipStream_t s);

// Measurement helper: n_blocks x 256 threads of independent bf16 MFMAs (iters x 8 per
// wave); out [n_blocks * 256] fp32 receives each thread's accumulator sum.
hipError_t launch_mfma_busy_loop(int n_blocks, int iters, float *out, hipStream_t s);

// ---- k_gemm.hip ---------------------------------------------------------------------
enum EpiMode { EPI_STORE = 0, EPI_QKV = 1, EPI_RESID = 2, EPI_SWIGLU = 3 };

struct Epi {
  int mode;
  void *out;            // STORE: [M][ldo] (out_dtype); RESID: float h [M][ldo]; SWIGLU: act
  int ldo;
  int out_dtype;        // AKVS_F32 / AKVS_BF16 for STORE / SWIGLU / QKV outputs
  // QKV: columns [0, hq_w) are q, [hq_w, hq_w+kv_w) k, the rest v; this GEMM's column 0
  // is logical column n_off.
  void *q_out, *k_out, *v_out;
  int n_off, hq_w, kv_w, hd;
  const int32_t *pos;   // row positions (nullptr: pos0 + row)
  int pos0;
  int kv_by_pos;        // k/v destination row = position (else = row)
  const float *rope;
  int rope_rows;
  int rope_base;        // position of the rotary table's first row
};

// C[M][N] = A[M][K] . B[N][K]^T with epilogue. Rows >= *m_dev (if given) are skipped.
// SWIGLU: N is the FFN width F; B has 2F rows (gate, then up). `part` (bf16 path, may be
// null) is a workspace of gemm_part_floats(M, N, K, mode) floats that lets grids too small
// to fill the GPU split K (partials summed in a fixed order by a second kernel). m_min is
// a lower bound on *m_dev known to the host: the split (and its second kernel) is only
// set up when some row count in [m_min, M] needs it.
hipError_t launch_gemm(const void *A, int lda, const void *B, int ldb, int M, int N, int K,
                       const int32_t *m_dev, int dtype, const Epi &epi, hipStream_t s,
                       float *part = nullptr, int m_min = 0);
// Second kernel of a K-split GEMM (same arguments as launch_gemm, launched right after it on
// the same stream); launches nothing when the first one cannot have split.
hipError_t launch_gemm_fixup(const void *A, int lda, const void *B, int ldb, int M, int N,
                             int K, const int32_t *m_dev, int dtype, const Epi &epi,
                             hipStream_t s, float *part = nullptr, int m_min = 0);
size_t gemm_part_floats(int M, int N, int K, int mode);
int gemm_cu_count();

// ---- k_attn.hip ---------------------------------------------------------------------
// With part_o / part_ml (bf16 path), the key range is split for parallelism:
// part_o [splits][rows][hq][hd] bf16 (each split's output over its own keys, normalised by
// its own sum; the buffer is typed float and needs half as many floats as elements),
// part_ml [splits][rows][hq][2] fp32 (max, sum), splits as below,
// lowered so that splits x rows stays within part_rows (what the buffers hold).
// row_base (device, may be null): rows start at row *row_base of q, pos and out.
hipError_t launch_attention(const void *q, const int32_t *pos, int pos0, int rows,
                            const int32_t *rows_dev, const void *k, const void *v, int n_keys,
                            int hq, int hkv, int hd, int dtype, void *out, float *part_o,
                            float *part_ml, long long part_rows, hipStream_t s,
                            const int32_t *row_base = nullptr, const int32_t *plan = nullptr);
// Plan of a split over the same rows (positions, row bound, live count, row_base as the
// launch_attention call that reads it; plan: kAttnPlanInts int32 of device memory, 16-byte
// aligned). Nothing is launched, and launch_attention ignores the plan, where the call's
// shape does not use one. The plan depends only on the rows' positions and n_keys: one
// plan serves every layer over the same rows.
constexpr int kAttnPlanInts = 4 * 65;
hipError_t launch_attention_plan(const int32_t *pos, int pos0, int rows, const int32_t *rows_dev,
                                 int n_keys, int hq, int hd, int dtype, long long part_rows,
                                 int32_t *plan, hipStream_t s, const int32_t *row_base = nullptr);
// number of key splits launch_attention uses for `rows` rows over n_keys keys
int attn_splits(int rows, int hq, int hkv, int n_keys);
// partial slots per row that the part_o / part_ml buffers of such a call should hold
int attn_part_splits(int rows, int hq, int hkv, int hd, int n_keys);
int attn_split_keys(int n_keys, int n_splits);

// ---- k_decode.hip -------------------------------------------------------------------
// Matrix-vector products of one token, y = W x (W [N][K], K a multiple of 8), item i of
// a launch = one pair of rows, with these epilogues:
//   GV_LOGITS  out_f32[n] = y[n]; part_val / part_idx [gemv_blocks(N)] get each block's
//              greedy best (largest value, lowest index), for launch_pick;
//   GV_RESID   out_f32[n] += y[n];
//   GV_SWIGLU  out[j] = silu(y[j]) * y[N/2 + j], j < N/2 (gate rows first);
//   GV_QKV     rows [q | k | v] of widths hq_w, kv_w, kv_w: q and k get the rotary map
//              with `rope` = the (cos, sin) row [hd/2] of the token's position, then
//              q -> q_out, k -> k_out, v -> v_out (out_dtype).
enum { GV_LOGITS = 0, GV_RESID = 1, GV_SWIGLU = 2, GV_QKV = 3 };
struct GemvEpi {
  int mode;
  float *out_f32;
  void *out;
  int out_dtype;
  void *q_out, *k_out, *v_out;
  int hq_w, kv_w, hd;
  const float2 *rope;
  float *part_val;
  int32_t *part_idx;
  // RMSNorm folded in front of the product: x is the fp32 residual row, each block forms
  // x * rstd * norm (rounded to the weight dtype) in LDS first; norm is in the weight dtype
  const void *norm;
  float eps;
};
int gemv_blocks(int N);
// Largest row width (elements) launch_gemv can normalise in LDS.
constexpr int GEMV_NORM_MAX = 16384;
hipError_t launch_gemv(const void *x, int x_dtype, const void *W, int w_dtype, int N, int K,
                       const GemvEpi &e, hipStream_t s);
// *out = index of the best of n (value, index) partials; -1 if none is a number.
// Attention of one new row (bf16, hd 64 or 128, hq / hkv <= 8) over n_keys cached keys:
// per (KV head, key chunk) partials part_o [n_chunks][hq][hd] and part_ml [n_chunks][hq][2]
// (fp32), merged into out [hq][hd] by a second kernel.
int decode_attn_chunks(int n_keys, int hkv, int *chunk_keys);
hipError_t launch_attention_decode(const void *q, const void *k, const void *v, int n_keys,
                                   int hq, int hkv, int hd, void *out, float *part_o,
                                   float *part_ml, hipStream_t s);
hipError_t launch_pick(const float *part_val, const int32_t *part_idx, int n, int32_t *out,
                       hipStream_t s);

}  // namespace akvs
