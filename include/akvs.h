/*
 * akvs.h - C ABI of the AgentKVShift reuse-prefill library for AMD MI355X (gfx950).
 *
 * The library computes the reuse prefill of "AgentKVShift: Efficient KV Cache Reuse
 * for Agentic Memory Systems": a query is prefilled on top of m memory units whose
 * per-layer K/V caches were computed once, each unit alone at position 0 (Sec. 3.1).
 * Cached keys are re-rotated to the unit's new offset, a small probe subset of each
 * unit plus the query is recomputed at every layer from the check layer on, each
 * unit's fresh-minus-reused offset is estimated on its probes, and every other token
 * is corrected by one weighted vector add (Sec. 3.3, Algorithm 1).
 *
 * Conventions shared by every entry point
 *  - Ownership: every tensor argument is a caller-owned DEVICE pointer, dense,
 *    row-major, 16-byte aligned, unless the argument says "host". Descriptor structs
 *    and chunk-length arrays are host memory read during the call only. The library
 *    never allocates, frees or keeps a pointer; scratch memory comes from a caller
 *    workspace sized by akvs_workspace_size / akvs_step_workspace_size (the one
 *    exception, akvs_decode_step_noalloc, uses a fixed device array of the library).
 *  - Streams: every call only enqueues work on `stream` and returns; buffers must stay
 *    alive until the stream has finished. akvs_chunk_meta and the query functions are
 *    host-only. Calls on different streams must not share output or workspace buffers.
 *  - Errors: an akvs_status is returned. Arguments are validated before anything is
 *    enqueued: an invalid call enqueues nothing and writes nothing. A HIP launch
 *    failure returns AKVS_EHIP. akvs_last_error() gives a message for the calling
 *    thread's last failure. No C++ exception crosses this interface.
 *  - Values held in device memory (token ids, positions, probe indices, chunk
 *    metadata) cannot be checked on the host. Kernels bound-check them and never
 *    read or write outside the buffers described here; an out-of-range value
 *    produces unspecified numbers in the affected rows, never a fault.
 *  - Determinism: no floating-point atomics; identical inputs on the same device give
 *    bitwise identical outputs.
 *  - dtypes: AKVS_F32 model = fp32 weights, activations and K/V; AKVS_BF16 model =
 *    bf16 weights and K/V, fp32 residual stream and accumulation. Quantised caches
 *    (AKVS_U4G64 / AKVS_U2G64 / AKVS_E4M3G64) are only valid as cache inputs of a bf16
 *    model.
 *
 * Layouts (L layers, D model width, Hq / Hkv heads, hd head dim, F FFN width,
 * kvw = Hkv*hd, T_c = sum of unit lengths, q = query length, T = T_c + q)
 *  - weights per layer [out][in]: w_qkv [(Hq+2Hkv)*hd][D] (q rows, then k, then v),
 *    w_o [D][Hq*hd], w_gate_up [2F][D] (gate rows first), w_down [D][F], norms [D];
 *    embed [V][D]; final_norm [D]. Weight dtype = model dtype.
 *  - unit caches k/v [L][T_c][Hkv][hd], units back to back in context order, token t
 *    of a unit stored as rotated at position t. Quantised: codes
 *    [L][T_c][Hkv][hd*bits/8] uint8 (low bits first: 4-bit element 2k is the low
 *    nibble of byte k, 2-bit element 4k is bits 0-1 of byte k) and meta
 *    [L][T_c][Hkv][hd/64][2] fp16 (scale, zero); x = scale*code + zero.
 *  - corrected / fresh caches [L][T][Hkv][hd], indexed by position.
 *  - rotary table [n_pos][hd/2][2] fp32 (cos, sin) of p * theta^(-2k/hd), rotate-half
 *    pairing of dimension k with k + hd/2.
 */
#ifndef AKVS_H
#define AKVS_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t akvs_status;
enum {
  AKVS_OK = 0,
  AKVS_EINVAL = 1,       /* null pointer, bad range, misaligned pointer          */
  AKVS_ESHAPE = 2,       /* inconsistent sizes                                   */
  AKVS_EDTYPE = 3,       /* dtype not valid for this argument / model            */
  AKVS_EUNSUPPORTED = 4, /* valid but not implemented (e.g. head_dim not 64/128) */
  AKVS_ENOSPACE = 5,     /* workspace too small                                  */
  AKVS_EHIP = 6          /* HIP runtime error while enqueueing                   */
};

enum { AKVS_F32 = 0, AKVS_BF16 = 1, AKVS_U4G64 = 2, AKVS_U2G64 = 3, AKVS_E4M3G64 = 4 };

/* akvs_reuse_cfg.flags */
enum {
  AKVS_F_NO_CORRECTION = 1u,       /* offsets forced to 0 (probes fresh, others as reused)   */
  AKVS_F_UNIT_WEIGHTS = 2u,        /* w = 1 instead of min(d, 1)                            */
  AKVS_F_FRESH_IF_RECOMPUTED = 4u, /* a token recomputed for either side takes fresh K and V */
  AKVS_F_NO_PREFIX_RECOMPUTE = 8u, /* stale reuse: no check layer; needs refresh_num == 0    */
  AKVS_F_GIVEN_PROBES = 16u,       /* probe sets come from the caller instead of top-b       */
  AKVS_F_PRE_ROPE_OFFSETS = 32u    /* key offsets taken before the rotary map: each probe's
                                      difference is rotated back by its position before the
                                      mean, the offset rotated to each corrected token's */
};

typedef struct akvs_model_cfg {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rope_theta, rms_eps;
  int32_t dtype; /* AKVS_F32 or AKVS_BF16 */
} akvs_model_cfg;

typedef struct akvs_layer_w {
  const void *attn_norm, *w_qkv, *w_o, *mlp_norm, *w_gate_up, *w_down;
} akvs_layer_w;

/* The retrieved units, the query and the method's parameters (Sec. 3.3, Alg. 1). */
typedef struct akvs_reuse_cfg {
  int32_t n_chunks;          /* m >= 1                                               */
  const int32_t *chunk_len;  /* host [m], every n_i >= 1                             */
  int32_t query_len;         /* q >= 1                                               */
  int32_t refresh_num, refresh_den; /* r = num/den in [0, 1]; b_i = ceil(num*n_i/den) */
  int32_t check_layer;       /* 0-based layer of the divergence check, < n_layers    */
  uint32_t flags;            /* AKVS_F_*                                             */
  int32_t refresh_v_num, refresh_v_den; /* value-side ratio (asymmetric K/V budgets);
                                           den 0: the key ratio for both sides       */
} akvs_reuse_cfg;

/* A unit cache: k, v in the cache layout above; k_meta / v_meta only when quantised. */
typedef struct akvs_cache {
  const void *k, *v;
  const void *k_meta, *v_meta;
  int32_t dtype; /* AKVS_F32 (f32 model), AKVS_BF16, AKVS_U4G64, AKVS_U2G64, AKVS_E4M3G64
                    (bf16 model) */
} akvs_cache;

/* Outputs of akvs_reuse_prefill. h_query, k_corr, v_corr are required; the others
 * may be NULL (then kept in the workspace only). */
typedef struct akvs_reuse_out {
  float *h_query;          /* [q][D] final-normed query rows                         */
  void *k_corr, *v_corr;   /* [L][T][Hkv][hd], model dtype                           */
  int32_t *probe_k, *probe_v; /* [sum b_i] global positions, per unit ascending (CSR) */
  float *d_k, *d_v;        /* [T_c] check-layer divergences                          */
  int32_t *rows;           /* [T] recomputed positions, ascending; first n_rows used  */
  int32_t *n_rows;         /* [1] number of recomputed rows M                        */
  int32_t kv_rows;         /* rows per layer of k_corr / v_corr: 0 means T; a larger
                              value leaves room for the tokens a decode step appends */
} akvs_reuse_out;

/* ---- library information ---------------------------------------------------- */
int32_t akvs_version(void);
const char *akvs_status_string(akvs_status s);
const char *akvs_last_error(void);

/* ---- host helpers -------------------------------------------------------------- */

/* Per-unit bookkeeping (Sec. 3.3: b = ceil(r n), exact integers). Host only.
 * meta_out (host, may be NULL): [2][m][4], table 0 for the keys and table 1 for the
 * values, row i = (start s_i, length n_i, budget b_i of that side, CSR offset of the
 * unit's probes of that side = b_0 + ... + b_{i-1}); the two tables differ only when the
 * value side has its own ratio. totals_out (host, may be NULL): [5] = (T_c, sum b_K,i,
 * row cap = sum min(n_i, b_K,i + b_V,i) + q, T, sum b_V,i). Device copies of meta_out
 * are the `chunk_meta` argument of the step entries below. */
akvs_status akvs_chunk_meta(const akvs_reuse_cfg *cfg, int32_t *meta_out, int32_t *totals_out);

/* Workspace bytes of akvs_reuse_prefill (cfg != NULL) or of akvs_full_prefill over
 * n_tokens tokens (cfg == NULL). Returns 0 for an invalid configuration. */
size_t akvs_workspace_size(const akvs_model_cfg *m, const akvs_reuse_cfg *cfg, int32_t n_tokens);
/* Workspace bytes of akvs_probe_qkv / akvs_probe_out_mlp over n_rows rows. */
size_t akvs_step_workspace_size(const akvs_model_cfg *m, int32_t n_rows);
/* Workspace bytes that let akvs_sparse_query_attention split the key range of n_rows rows
 * over n_keys keys (the launch configuration of the reuse prefill: the split partials and,
 * for few rows, a plan of the split made on the device from the positions); 0 when that
 * call would not split (fp32 models, or enough row tiles to fill the GPU). */
size_t akvs_attention_workspace_size(const akvs_model_cfg *m, int32_t n_rows, int32_t n_keys);

/* ---- step entries ---------------------------------------------------------------- */

/* Rotary table for positions 0..n_pos-1 (Sec. 2: reused states are moved to their new
 * positions by adjusting their positional embedding; rotary embeddings, rotate-half form, are
 * this library's reading of the decoders of Sec. 4.1, and every re-rotation, probe QKV
 * projection and pre-RoPE offset reads this table):
 * table[p][k] = (cos, sin)(p * theta^(-2k/hd)), angles and their cos/sin in fp64, stored
 * rounded to fp32. table: [n_pos][hd/2][2], caller-owned device memory, 16-byte aligned;
 * n_pos = 0 writes nothing. Errors: EINVAL (n_pos < 0, hd odd or outside [2, 1024],
 * theta <= 0, null or misaligned table), EHIP. */
akvs_status akvs_rope_table(int32_t n_pos, int32_t head_dim, float rope_theta, float *table,
                            hipStream_t stream);

/* Re-encode cached keys at a new offset (Sec. 2, positional re-encoding of reused
 * states): k_dst[t] = Rot(pos_delta[t]) deq(k_src[t]), v_dst[t] = deq(v_src[t]).
 * src: n_tokens rows of [Hkv][hd] in the cache layout of src->dtype (one layer);
 * pos_delta: device [n_tokens], 0 <= delta < rope_rows; rope: akvs_rope_table output
 * with rope_rows rows. dst_dtype: AKVS_F32 (f32 cache) or AKVS_BF16. */
akvs_status akvs_rerotate_keys(const akvs_cache *src, int32_t n_tokens, int32_t n_kv_heads,
                               int32_t head_dim, const int32_t *pos_delta, const float *rope,
                               int32_t rope_rows, void *k_dst, void *v_dst, int32_t dst_dtype,
                               hipStream_t stream);

/* Check-layer divergence (Sec. 3.3 display equation): d_k[t] = || k_fresh[t] -
 * Rot(pos_delta[t]) deq(k_cached[t]) ||_2 over all Hkv*hd components, d_v likewise
 * without rotation; fp32 sums. fresh: [n_tokens][Hkv][hd] of fresh_dtype (F32/BF16);
 * cache: one layer as in akvs_rerotate_keys; pos_delta may be NULL (no rotation). */
akvs_status akvs_check_divergence(const void *k_fresh, const void *v_fresh, int32_t fresh_dtype,
                                  const akvs_cache *cache, int32_t n_tokens, int32_t n_kv_heads,
                                  int32_t head_dim, const int32_t *pos_delta, const float *rope,
                                  int32_t rope_rows, float *d_k, float *d_v, hipStream_t stream);

/* Probe selection (Sec. 3.3 "Probe selection"; Alg. 1): per unit i, S_K,i = the b_i
 * tokens of largest d_k (equal values: the earlier token first), S_V,i likewise;
 * weights w = min(d, 1) (1 with AKVS_F_UNIT_WEIGHTS). With AKVS_F_GIVEN_PROBES the
 * sets are read from probe_k / probe_v (as written below) instead. Writes
 *  probe_k [sum b_K,i], probe_v [sum b_V,i]: global positions, ascending within each
 *   unit, unit i at the CSR offset of its side's table (meta[0][i][3] / meta[1][i][3]);
 *  flags [T_c] uint8: bit0 = in S_K, bit1 = in S_V;  w_k, w_v [T_c] fp32;
 *  chunk_rows [m]: |S_K,i u S_V,i|;
 *  rows [row cap]: recomputed positions R = (u_i S_K,i u S_V,i) u query, ascending;
 *  n_rows [1]: |R|;  fresh_row [T]: index in R of each position, -1 if not recomputed.
 * chunk_meta: device copy of akvs_chunk_meta's meta_out. d_k, d_v must be finite. A
 * probe array may be NULL when its side's budgets are all 0. */
akvs_status akvs_select_probes(const float *d_k, const float *d_v, const akvs_reuse_cfg *cfg,
                               const int32_t *chunk_meta, int32_t *probe_k, int32_t *probe_v,
                               float *w_k, float *w_v, uint8_t *flags, int32_t *chunk_rows,
                               int32_t *rows, int32_t *n_rows, int32_t *fresh_row,
                               hipStream_t stream);

/* Probe-row projections (Alg. 1, recompute of the probe rows): x = RMSNorm(h[r]) *
 * attn_norm; [q|k|v] = x W_qkv^T; RoPE on q and k at positions[r]. h: [n_rows][D] fp32;
 * positions: device [n_rows] (each < rope_rows); q: [n_rows][Hq][hd], k_fresh / v_fresh:
 * [n_rows][Hkv][hd] in the model dtype. */
akvs_status akvs_probe_qkv(const float *h, int32_t n_rows, const int32_t *positions,
                           const akvs_model_cfg *m, const akvs_layer_w *lw, const float *rope,
                           int32_t rope_rows, void *q, void *k_fresh, void *v_fresh, void *ws,
                           size_t ws_bytes, hipStream_t stream);

/* Per-unit offsets of one layer (Sec. 3.3 "Mean estimation"; Alg. 1):
 * mu_k[i] = (1/b_i) sum_{j in S_K,i} (k_fresh[fresh_row[j]] - Rot(s_i) deq(k_cached[j])),
 * mu_v likewise without rotation; 0 when b_i = 0 or with AKVS_F_NO_CORRECTION. With
 * AKVS_F_PRE_ROPE_OFFSETS each key term is first rotated back by -j (the offset is then
 * a pre-RoPE vector). Probe terms are summed in ascending position order in fp32. k_fresh / v_fresh: [rows][Hkv][hd]
 * model dtype; cache: one layer; mu_k, mu_v: [m][Hkv][hd] fp32. */
akvs_status akvs_chunk_offset(const void *k_fresh, const void *v_fresh, const int32_t *fresh_row,
                              const akvs_cache *cache, const akvs_reuse_cfg *cfg,
                              const int32_t *chunk_meta, const int32_t *probe_k,
                              const int32_t *probe_v, const akvs_model_cfg *m, const float *rope,
                              int32_t rope_rows, float *mu_k, float *mu_v, hipStream_t stream);

/* Corrected cache of one layer (Alg. 1 inner loop; Sec. 3.3 "AgentKVShift correction").
 * For a unit token j of unit i: k_corr[j] = k_fresh[fresh_row[j]] if j in S_K,i (any
 * recomputed j with AKVS_F_FRESH_IF_RECOMPUTED), else Rot(s_i) deq(k_cached[j]) +
 * w_k[j] mu_k[i] (w_k[j] Rot(j) mu_k[i] with AKVS_F_PRE_ROPE_OFFSETS); v_corr likewise
 * with S_V and no rotation. Query positions T_c..T-1
 * take their fresh rows. k_corr, v_corr: [T][Hkv][hd] model dtype (one layer). */
akvs_status akvs_apply_correction(const akvs_cache *cache, const float *mu_k, const float *mu_v,
                                  const float *w_k, const float *w_v, const uint8_t *flags,
                                  const void *k_fresh, const void *v_fresh,
                                  const int32_t *fresh_row, const akvs_reuse_cfg *cfg,
                                  const int32_t *chunk_meta, const akvs_model_cfg *m,
                                  const float *rope, int32_t rope_rows, void *k_corr,
                                  void *v_corr, hipStream_t stream);

/* Attention of sparse query rows over a full key range (Alg. 1 recompute of the probe
 * rows against the whole corrected context): row r at position positions[r] attends
 * to keys 0..positions[r] (< n_keys) with scores q.k/sqrt(hd), fp32 softmax, query
 * head h reading KV head h/(Hq/Hkv). q: [n_rows][Hq][hd]; k, v: [n_keys][Hkv][hd];
 * out: [n_rows][Hq*hd]; all model dtype. positions must be ascending. ws (may be NULL)
 * of ws_bytes >= akvs_attention_workspace_size lets the call split the key range and
 * merge the parts, as the reuse prefill does; a non-NULL ws that is too small is
 * AKVS_ENOSPACE. */
akvs_status akvs_sparse_query_attention(const void *q, const int32_t *positions, int32_t n_rows,
                                        const void *k, const void *v, int32_t n_keys,
                                        const akvs_model_cfg *m, void *out, void *ws,
                                        size_t ws_bytes, hipStream_t stream);

/* Rest of the probe rows' layer (Algorithm 1, "recompute fresh KV for S_K u S_V at layer
 * l": the fresh K/V of the next layer need these rows' hidden states carried through this
 * layer's attention output and MLP; Sec. 3.3): h += attn_out W_o^T;
 * x = RMSNorm(h) * mlp_norm; h += (silu(x W_gate^T) * (x W_up^T)) W_down^T.
 * h: [n_rows][D] fp32 (updated in place); attn_out: [n_rows][Hq*hd] model dtype. */
akvs_status akvs_probe_out_mlp(float *h, int32_t n_rows, const void *attn_out,
                               const akvs_model_cfg *m, const akvs_layer_w *lw, void *ws,
                               size_t ws_bytes, hipStream_t stream);

/* Group-64 quantiser of a cache (Sec. 4.5 composition with KV quantisation). For each
 * group of 64 head-dim elements:
 *   bits 2 / 4 (AKVS_U2G64 / AKVS_U4G64, asymmetric integer codes): zero = fp16(min),
 *     scale = fp16((max-min) / (2^bits - 1)) computed in fp32,
 *     code = clamp(rne((x - zero) / scale), 0, 2^bits - 1) (0 when scale == 0);
 *   bits 8 (AKVS_E4M3G64, FP8 E4M3 codes): scale = fp16(max|x| / 448) computed in fp32,
 *     zero = 0, code = E4M3 of clamp(x / scale, -448, 448) rounded half to even (OCP FP8
 *     E4M3: bias 7, no infinity, 448 the largest finite value; 0 when scale == 0).
 * x: [n_rows][hd] of x_dtype (F32 or BF16), hd a multiple of 64; codes:
 * [n_rows][hd*bits/8]; meta: [n_rows][hd/64][2] fp16 (scale, zero). */
akvs_status akvs_quantize_cache(const void *x, int32_t x_dtype, int32_t n_rows, int32_t head_dim,
                                int32_t bits, uint8_t *codes, void *meta, hipStream_t stream);

/* ---- whole-procedure entries -------------------------------------------------------- */

/* Reuse prefill (Algorithm 1 over all layers). tokens: device [T] ids (units in order,
 * then the query), each in [0, vocab). lw: host array of n_layers layer weight sets.
 * Layers before check_layer are computed for every token; from check_layer on only
 * R = probes u query is recomputed and every unit token takes its corrected state.
 * With AKVS_F_GIVEN_PROBES, out->probe_k / out->probe_v must hold the sets on entry. */
akvs_status akvs_reuse_prefill(const int32_t *tokens, const void *embed, const akvs_layer_w *lw,
                               const void *final_norm, const akvs_model_cfg *m,
                               const akvs_reuse_cfg *cfg, const akvs_cache *cache,
                               const akvs_reuse_out *out, void *ws, size_t ws_bytes,
                               hipStream_t stream);

/* Batched reuse prefill (the paper's batch axis, Sec. 4.4 / Table 3: B requests served
 * together). Request b is exactly the call akvs_reuse_prefill(tokens[b], ..., &cfgs[b],
 * &caches[b], &outs[b]) — its own units, query, unit caches, outputs and probe sets —
 * but from the check layer on the recomputed rows of all requests form one row block,
 * so every projection GEMM reads its weights once per layer for the whole batch;
 * offsets, correction and attention stay per request. tokens, cfgs, caches and outs are
 * host arrays of `batch` entries (device pointers inside, as for akvs_reuse_prefill).
 * Every cfg must use the same check_layer and AKVS_F_NO_PREFIX_RECOMPUTE setting
 * (AKVS_EINVAL otherwise). ws: akvs_batch_workspace_size bytes. */
akvs_status akvs_reuse_prefill_batch(const int32_t *const *tokens, int32_t batch,
                                     const void *embed, const akvs_layer_w *lw,
                                     const void *final_norm, const akvs_model_cfg *m,
                                     const akvs_reuse_cfg *cfgs, const akvs_cache *caches,
                                     const akvs_reuse_out *outs, void *ws, size_t ws_bytes,
                                     hipStream_t stream);
/* Workspace bytes of akvs_reuse_prefill_batch (0 for an invalid configuration). */
size_t akvs_batch_workspace_size(const akvs_model_cfg *m, const akvs_reuse_cfg *cfgs,
                                 int32_t batch);

/* Full prefill (the no-reuse baseline; also the standalone caching of a unit with
 * pos0 = 0, Sec. 3.1). tokens: device [n] ids at positions pos0..pos0+n-1. h_out:
 * [n][D] fp32 final-normed hidden states (may be NULL); k_out, v_out: [L][n][Hkv][hd]
 * model dtype (post-RoPE keys). */
akvs_status akvs_full_prefill(const int32_t *tokens, int32_t n_tokens, int32_t pos0,
                              const void *embed, const akvs_layer_w *lw, const void *final_norm,
                              const akvs_model_cfg *m, float *h_out, void *k_out, void *v_out,
                              void *ws, size_t ws_bytes, hipStream_t stream);

/* ---- first decode step over the corrected caches -------------------------------------
 * The consumer of a reuse prefill: the next token is predicted from the last final-normed
 * query row, then generated tokens run through every layer attending to the corrected
 * keys and values (Sec. 3.1: the reused states serve the generation that follows). The
 * output embedding w_out is [vocab][D] in the model dtype; NULL means tied to the input
 * embedding (as in the 3B-class decoders the paper evaluates). Greedy pick: the largest
 * logit, equal values resolved to the lowest index, -1 if no logit is a number. */

/* Workspace of akvs_decode_step with n_past cached tokens (also enough for akvs_lm_head
 * when n_past >= 0). 0 for an invalid model. */
size_t akvs_decode_workspace_size(const akvs_model_cfg *m, int32_t n_past);

/* logits[r][:] = h[r] . w_out^T and tokens[r] = greedy pick, r < n_rows. h: device
 * [n_rows][D] fp32 final-normed rows (e.g. the last row of h_query); logits (device
 * [n_rows][vocab] fp32) or tokens (device [n_rows]) may be NULL, not both. */
akvs_status akvs_lm_head(const float *h, int32_t n_rows, const void *w_out,
                         const akvs_model_cfg *m, float *logits, int32_t *tokens, void *ws,
                         size_t ws_bytes, hipStream_t stream);

/* One decode step: token (device [1]) at position n_past. k_cache, v_cache: device
 * [L][cache_rows][Hkv][hd] model dtype, rows 0..n_past-1 valid (e.g. the k_corr / v_corr
 * of a reuse prefill written with kv_rows = cache_rows); the step writes the token's
 * post-RoPE key and value to row n_past of every layer. Outputs logits (device [vocab]
 * fp32, may be NULL) and next_token (device [1], may be NULL). Errors: EINVAL for
 * n_past < 0 or cache_rows <= n_past, null or misaligned pointers; ENOSPACE. */
akvs_status akvs_decode_step(const int32_t *token, int32_t n_past, const void *embed,
                             const akvs_layer_w *lw, const void *final_norm, const void *w_out,
                             const akvs_model_cfg *m, void *k_cache, void *v_cache,
                             int32_t cache_rows, float *logits, int32_t *next_token, void *ws,
                             size_t ws_bytes, hipStream_t stream);

/* ---- decode step without allocation ---------------------------------------------------
 * For callers that cannot allocate device memory or pass a workspace: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc. akvs_decode_step_noalloc
 * is akvs_decode_step (same arguments, same kernels, identical results) with the workspace
 * taken from a device array inside the library of AKVS_NOALLOC_SCRATCH_BYTES bytes, which
 * every device that runs it holds until the process ends. The call itself allocates nothing
 * and frees nothing; its first call on a device looks up that device's array address.
 * Errors: AKVS_ENOSPACE when akvs_decode_workspace_size(m, n_past) exceeds
 * AKVS_NOALLOC_SCRATCH_BYTES (the attention partials grow with n_past: about 200K past
 * tokens for the 32B-class shape); AKVS_EINVAL when `stream` belongs to a device other
 * than the calling thread's current one; otherwise as akvs_decode_step. All calls on one
 * device share that device's array: calls that overlap in time on one device (on different
 * streams, or from several threads without ordering) race on it and give unspecified
 * results. Calls ordered on one stream are safe; the array keeps the last call's contents,
 * none of which a later call reads before writing it. */
#define AKVS_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
akvs_status akvs_decode_step_noalloc(const int32_t *token, int32_t n_past, const void *embed,
                                     const akvs_layer_w *lw, const void *final_norm,
                                     const void *w_out, const akvs_model_cfg *m, void *k_cache,
                                     void *v_cache, int32_t cache_rows, float *logits,
                                     int32_t *next_token, hipStream_t stream);

/* ---- kernel timing -------------------------------------------------------------------
 * akvs_profile_enable(mask): for every kernel class whose bit (1 << class) is set in
 * mask, the library brackets each launch of that class with a pair of HIP events
 * recorded on the launch stream and accumulates the number of launches and the summed
 * event time (0 disables). akvs_profile_read waits for the recorded events, returns the
 * class totals and clears that class. Process-wide state, meant for a single
 * benchmarking thread. */
enum {
  AKVS_K_GEMM = 0, AKVS_K_ATTENTION = 1, AKVS_K_CORRECTION = 2, AKVS_K_OFFSET = 3,
  AKVS_K_DIVERGENCE = 4, AKVS_K_SELECT = 5, AKVS_K_NORM = 6, AKVS_K_OTHER = 7,
  AKVS_K_GEMV = 8, AKVS_K_NCLASSES = 9
};
akvs_status akvs_profile_enable(int32_t class_mask);
akvs_status akvs_profile_read(int32_t kernel_class, int64_t *launches, double *total_ms);

/* ---- counter calibration ----------------------------------------------------------------
 * akvs_mfma_busy_loop: not part of the method; the reference point for hardware counters
 * of matrix-core use and for the MFMA rate the chip sustains. Launches n_blocks blocks of
 * 256 threads in which every wave issues iters (rounded up to even) x 8 independent
 * 32x32x16 bf16 MFMAs on random operands that change from one MFMA to the next, and
 * nothing else (the matrix cores of every SIMD it occupies stay busy), then writes one
 * fp32 per thread to out (device
 * [n_blocks * 256], caller-owned, 16-byte aligned). Asynchronous on stream. Errors:
 * EINVAL for negative sizes, a null or misaligned out (with n_blocks > 0); EHIP. */
akvs_status akvs_mfma_busy_loop(int32_t n_blocks, int32_t iters, float *out, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* AKVS_H */
