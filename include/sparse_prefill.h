/*
 * sparse_prefill.h — C ABI of the MI355X (gfx950) causal top-k sparse GQA
 * prefill library.
 *
 * The library computes, for one grouped-query-attention layer, the sparse
 * prefill path of "How Much Dense Attention is Necessary? Oracle-Guided
 * Sparse Prefill for Full/GQA Layers in Hybrid Long-Context Models":
 *
 *   indexer mode (Algorithm 2, scoring, selection and sparse prefill):
 *     sp_indexer_scores -> sp_topk_select -> sp_sparse_gqa_attn
 *   oracle mode (Algorithm 1, dense pass, selection and restricted recomputation):
 *     sp_dense_attn (normalisers) -> sp_oracle_support -> sp_topk_select
 *     -> sp_sparse_gqa_attn
 *   dense baseline (Section 3):
 *     sp_dense_attn
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Indices are 0-based. S = seq_len, Hq query heads, Hkv KV heads,
 * G = Hq/Hkv, query head h reads KV head g(h) = floor(h/G) (contiguous
 * groups), d = head_dim, d_idx = index_dim, k = topk, b = block_q (the
 * selection block size b_sel), R = ceil(S/b) selection blocks; block r
 * holds queries t0_r = r*b ... t1_r = min(r*b+b, S)-1.
 *
 * Layouts (all contiguous, row-major, element type = problem dtype unless
 * stated):
 *   q, o          [S, Hq,  d]
 *   k, v          [S, Hkv, d]
 *   q_idx, k_idx  [S, d_idx]
 *   lse           [S, Hq]  float32
 *   scores, mass  [R, S]   float32; row r is valid for columns s <= t1_r
 *                          only: later columns are never written nor read
 *   idx           [R, k]   int32; ascending positions, then -1 sentinels;
 *                          one row serves every query of block r and every
 *                          KV head
 * With head_axis = 1 (one support per KV group) mass and idx gain a leading
 * KV-group axis: mass [Hkv, R, S], idx [Hkv, R, k]; sp_topk_select then
 * takes scores [Hkv, R, S].
 *
 * Memory and ownership: every pointer is a DEVICE pointer allocated and
 * owned by the caller, 16-byte aligned, and inputs never alias outputs.
 * The library allocates nothing. Its only mutable global state is a set of
 * per-device caches filled on first use and never invalidated: the device
 * architecture, the compute-unit count, and the resident-workgroup count
 * of each persistent kernel instance (all written atomically, so calls from
 * several host threads are safe).
 *
 * Execution: each call validates its arguments on the host before any HIP
 * call (so validation needs no GPU), then enqueues its kernels on `stream`
 * and returns without synchronising. Faults inside a kernel surface at the
 * caller's next synchronisation.
 *
 * Errors: each entry point returns SP_OK or a negative sp_status; on error
 * nothing has been enqueued.
 */
#ifndef SPARSE_PREFILL_H_
#define SPARSE_PREFILL_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SP_VERSION 10000 /* 1.0.0 */

typedef enum sp_status {
  SP_OK = 0,
  SP_ERR_NULL = -1,        /* a required pointer is NULL */
  SP_ERR_SHAPE = -2,       /* inconsistent sizes (e.g. Hq % Hkv != 0, k < 1) */
  SP_ERR_UNSUPPORTED = -3, /* valid but not built: head_dim, dtype, causal=0,
                              k or v of 4 GiB or more */
  SP_ERR_WORKSPACE = -4,   /* workspace smaller than sp_workspace_bytes */
  SP_ERR_ALIGN = -5,       /* a pointer is not 16-byte aligned */
  SP_ERR_NO_DEVICE = -6,   /* no HIP device is usable */
  SP_ERR_ARCH = -7,        /* current device is not gfx950 */
  SP_ERR_HIP = -8          /* a HIP launch failed */
} sp_status;

enum { SP_DTYPE_F32 = 0, SP_DTYPE_BF16 = 1 };
enum { SP_AGG_MAX = 0, SP_AGG_SUM = 1 };
enum { SP_OP_DENSE = 0, SP_OP_ORACLE = 1, SP_OP_INDEXER = 2, SP_OP_TOPK = 3,
       SP_OP_SPARSE = 4, SP_OP_KL = 5, SP_OP_PROJECT = 6, SP_OP_INDEXER_TOPK = 7 };

/*
 * One GQA layer's sparse-prefill problem (Section 3: S, Hq, Hkv, d_h, the
 * map g; Section 3 support granularity: b_sel; Section 3 restricted
 * attention: |S_t| <= k; Section 6.3: d_idx).
 */
typedef struct sp_problem {
  int32_t seq_len;      /* S >= 1; k and v ([S,Hkv,d]) each below 4 GiB */
  int32_t num_q_heads;  /* Hq >= 1, a multiple of num_kv_heads */
  int32_t num_kv_heads; /* Hkv >= 1 */
  int32_t head_dim;     /* d: 64, 128 or 256 (Section 6.3: d = d_idx = 256
                           for some backbones) */
  int32_t index_dim;    /* d_idx: 64, 128 or 256 (indexer calls only) */
  int32_t topk;         /* k >= 1; k >= t1_r+1 keeps every causal key */
  int32_t block_q;      /* b >= 1; 1 = per-query support */
  int32_t causal;       /* must be 1: the paper's attention is causal */
  int32_t local_window; /* W in [0, k]: the W most recent positions of each
                           block are always selected, counted inside k */
  int32_t agg;          /* SP_AGG_MAX (Section 4.2) or SP_AGG_SUM */
  int32_t relu;         /* 1: ReLU on indexer scores (Section 6.3); 0: raw */
  int32_t dtype;        /* SP_DTYPE_F32 or SP_DTYPE_BF16 for q,k,v,o,q_idx,k_idx */
  float attn_scale;     /* 0 => 1/sqrt(d) (Section 3); otherwise finite and
                           positive: a negative value is SP_ERR_SHAPE */
  float index_scale;    /* 0 => 1/sqrt(d_idx) (Section 6.3) */
  int32_t head_axis;    /* support granularity on the head axis (Section 3):
                           0: one head-averaged token support S_t shared by all
                              query heads (mass and tables [R, ...]);
                           1: one support S_{t,r} per KV group r, used by the G
                              query heads of the group (mass and tables
                              [Hkv, R, ...]). The indexer is head-collapsed and
                              takes 0 only. */
  int32_t q_offset;     /* chunked prefill: the call covers query positions
                           q_offset .. S-1 of a sequence whose keys are 0 .. S-1
                           (S = seq_len). q, o, lse and q_idx then hold the
                           S - q_offset chunk rows; k, v and k_idx all S rows;
                           selection blocks are counted from q_offset (which
                           must be a multiple of block_q), so R = ceil((S -
                           q_offset) / b) and row r holds positions
                           q_offset + r*b ... Used by sp_dense_attn,
                           sp_indexer_scores, sp_topk_select and the sparse
                           attention calls; 0 elsewhere. */
} sp_problem;

/*
 * Dense causal GQA attention (Section 3, first equation; Algorithm 1, dense scores and normalisers).
 *   o[t,h]   = sum_{s<=t} softmax_{s'<=t}(attn_scale * <q[t,h], k[s',g(h)]>)_s v[s,g(h)]
 *   lse[t,h] = log sum_{s<=t} exp(attn_scale * <q[t,h], k[s,g(h)]>)
 * o may be NULL when lse is given: only the softmax normalisers are
 * computed (what the oracle needs). lse may be NULL. Both NULL is
 * SP_ERR_NULL. Fields used: seq_len, heads, head_dim, causal, dtype,
 * attn_scale.
 */
int sp_dense_attn(const sp_problem *p, const void *q, const void *k, const void *v,
                  void *o, float *lse, hipStream_t stream);

/*
 * Attention-mass oracle scores (Section 4.1 head-averaged mass; Section 4.2
 * block max; Algorithm 1, head-averaged probabilities):
 *   P_t(s)    = (1/Hq) sum_h exp(attn_scale * <q[t,h], k[s,g(h)]> - lse[t,h]),  s <= t
 *   mass[r,s] = AGG_{t in block r, t >= s} P_t(s),  s <= t1_r
 * lse must come from sp_dense_attn on the same q, k and problem. AGG is
 * `agg` (the paper's rule is max); with block_q = 1 mass[t,s] = P_t(s).
 * head_axis = 1: mass[j,r,s] uses P_{t,j}(s) = (1/G) sum over the G heads of
 * KV group j (the per-group support S_{t,r} of Section 3).
 */
int sp_oracle_support(const sp_problem *p, const void *q, const void *k, const float *lse,
                      float *mass, hipStream_t stream);

/*
 * Head-collapsed indexer scores (Section 6.3 equation for z; Algorithm 2,
 * candidate scoring):
 *   z[t,s]      = ReLU(index_scale * <q_idx[t], k_idx[s]>),  s <= t  (no ReLU if relu=0)
 *   scores[r,s] = AGG_{t in block r, t >= s} z[t,s],  s <= t1_r
 * q_idx/k_idx are the indexer vectors after key normalisation, RoPE and
 * any query scale (Algorithm 2, query scale).
 */
int sp_indexer_scores(const sp_problem *p, const void *q_idx, const void *k_idx,
                      float *scores, hipStream_t stream);

/*
 * Top-k support selection (Section 4.1 TopK; Section 4.2; Algorithm 1,
 * selection and restricted recomputation; Algorithm 2, selection and sparse
 * GQA prefill). For block r with L = t1_r+1 causal positions:
 *   L <= k : idx[r] = 0..L-1, then -1;
 *   L >  k : the Wf = min(local_window, k) positions t1_r-Wf+1..t1_r are
 *            forced; the other k-Wf are the first positions of 0..L-Wf-1
 *            in the order (score descending, position ascending), with
 *            -0.0 treated as +0.0.
 * Each row is written ascending. NaN scores give an unspecified (but
 * in-bounds) selection. workspace may be NULL when sp_workspace_bytes
 * reports 0 for SP_OP_TOPK (it does in this version).
 */
int sp_topk_select(const sp_problem *p, const float *scores, int32_t *idx, void *workspace,
                   size_t workspace_bytes, hipStream_t stream);

/*
 * Sparse GQA attention over the shared supports (Section 3, second
 * equation; Section 4.2 per-query causal mask; Algorithm 1, restricted recomputation).
 * Query t of block r = t/b, head h, uses U = { s in idx[r,:] : 0 <= s <= t }:
 *   o[t,h] = sum_{s in U} softmax_U(attn_scale * <q[t,h], k[s,g(h)]>)_s v[s,g(h)]
 * and o[t,h] = 0 when U is empty. Entries < 0 or >= S are skipped (they are
 * sentinels); positions within a row must be distinct. The order of a row
 * does not change the result beyond rounding. head_axis = 1: head h uses the
 * table idx[g(h), r, :] of its KV group instead.
 */
int sp_sparse_gqa_attn(const sp_problem *p, const void *q, const void *k, const void *v,
                       const int32_t *idx, void *o, hipStream_t stream);

/*
 * Sparse GQA attention reading K and V from a paged cache (Section 6.4: the
 * serving path gathers the selected support inside the attention kernel, from
 * a paged KV cache). Same result as sp_sparse_gqa_attn on the contiguous K, V
 * with K[s] = k_pages[page_table[s / page_size], s % page_size]:
 *   k_pages, v_pages: device [num_pages, page_size, Hkv, d] (problem dtype),
 *                     each below 4 GiB;
 *   page_table:       device int32 [ceil(S / page_size)]: the physical page of
 *                     each logical page of the sequence. A selected position
 *                     whose page entry is outside [0, num_pages) is skipped
 *                     like a sentinel (nothing outside the cache is read).
 * Everything else (q, idx, o, head_axis, block_q) as sp_sparse_gqa_attn.
 */
int sp_sparse_gqa_attn_paged(const sp_problem *p, const void *q, const void *k_pages,
                             const void *v_pages, const int32_t *page_table, int32_t page_size,
                             int32_t num_pages, const int32_t *idx, void *o,
                             hipStream_t stream);

/*
 * Fused per-query indexer scoring and top-k (Section 6.3 score equation;
 * Section 6.4 fused path and Algorithm 2, scoring, selection and sparse prefill with b_sel = 1; Section 4.1
 * TopK): idx[t,:] = the top-k positions of z[t,s] = ReLU?(index_scale *
 * <q_idx[t], k_idx[s]>) over s <= t, selected exactly as sp_topk_select does
 * on those scores (forced window of min(W,k) most recent positions, then
 * score descending / position ascending; ascending rows, -1 padded), without
 * storing the S x S score matrix: scores are recomputed on the matrix cores
 * in each pass of an 8-bit radix select.
 * Requires block_q = 1, dtype bf16, index_dim 64/128/256, seq_len <= 65535,
 * index_scale >= 0; otherwise SP_ERR_UNSUPPORTED. q_idx, k_idx: device bf16
 * [S, d_idx]; idx: device int32 [S, k] (output). workspace: device memory of
 * at least sp_workspace_bytes(p, SP_OP_INDEXER_TOPK) bytes (about
 * S * (512 * ceil(S/4096) + 144) bytes), caller-owned, 16-byte aligned,
 * contents undefined on entry and exit; SP_ERR_WORKSPACE if smaller.
 * Stream-ordered; several kernels are launched; nothing is allocated.
 */
int sp_indexer_topk(const sp_problem *p, const void *q_idx, const void *k_idx, int32_t *idx,
                    void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * sp_indexer_topk without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc). Same operation, arguments,
 * output and requirements as sp_indexer_topk; the scratch lives in a static
 * device array of the library, 64 MiB per GPU (SP_INDEXER_TOPK_STATIC_BYTES),
 * held from the library's first use on that GPU until the process ends.
 * Problems whose sp_workspace_bytes(p, SP_OP_INDEXER_TOPK) exceeds it
 * (seq_len above about 20480) return SP_ERR_WORKSPACE before anything is
 * enqueued. Nothing is allocated. Every call on one GPU shares that GPU's
 * array: calls that may overlap on one GPU (on different streams, or from
 * several host threads without ordering) race and must be serialised by the
 * caller; calls ordered on one stream are safe.
 */
#define SP_INDEXER_TOPK_STATIC_BYTES (64u << 20)
int sp_indexer_topk_noalloc(const sp_problem *p, const void *q_idx, const void *k_idx,
                            int32_t *idx, hipStream_t stream);

/*
 * Head-collapsed indexer front end (Section 6.3, the projection equations
 * and the score equation's RoPE; Algorithm 2, indexer projection and its key normalisation, RoPE and query scale): for token t at
 * position pos0 + t, with x_t = x[t,:],
 *   q_idx[t] = RoPE(W_Q x_t, pos0 + t),
 *   k_idx[t] = RoPE(LN(W_K x_t), pos0 + t),
 *   LN(a)    = (a - mean(a)) / sqrt(var(a) + ln_eps) * gamma + beta   over the d_idx entries,
 *   RoPE(a, p): each pair (a[c], a[c + d_idx/2]), c < d_idx/2, is rotated by the
 *              angle p * rope_theta^(-2c/d_idx):
 *              (a[c] cos - a[c+d_idx/2] sin, a[c+d_idx/2] cos + a[c] sin).
 * The 1/sqrt(d_idx) query scale is not applied here (sp_indexer_scores
 * applies index_scale). The outputs are the q_idx, k_idx inputs of
 * sp_indexer_scores. x: device bf16 [S, d_model], d_model a multiple of 64;
 * w_q, w_k: device bf16 [d_idx, d_model] (row c projects onto entry c);
 * gamma, beta: device fp32 [d_idx]; q_idx, k_idx: device bf16 [S, d_idx]
 * (outputs). pos0 >= 0 (a chunk of a longer sequence starts at pos0),
 * rope_theta > 0, ln_eps >= 0. Fields used: seq_len, index_dim, dtype (must be
 * SP_DTYPE_BF16). Caller-owned memory, stream-ordered, allocates nothing.
 */
int sp_indexer_project(const sp_problem *p, int32_t d_model, int32_t pos0, float rope_theta,
                       float ln_eps, const void *x, const void *w_q, const void *w_k,
                       const float *gamma, const float *beta, void *q_idx, void *k_idx,
                       hipStream_t stream);

/*
 * KL distillation objective of the indexer and its gradient (Section 6.2,
 * the loss equation): for supervised query rows t_i = rows[i], i < n_rows,
 *   kl[i]  = KL(P_i || softmax(z_i)) = sum_{s<=t_i} P_i(s) (log P_i(s) - z_i(s)) + LSE_i * sum_{s<=t_i} P_i(s),
 *   LSE_i  = log sum_{s<=t_i} exp z_i(s)   (the softmax runs over valid causal keys only),
 *   *loss  = (1/n_rows) sum_i kl[i],
 *   grad_z[i,s] = d loss / d z_i(s) = (softmax(z_i)(s) * sum P_i - P_i(s)) / n_rows for s <= t_i,
 *                 0 for t_i < s < S,
 * with 0 * log 0 = 0 and P taken as given (a head-averaged mass row, the
 * teacher of Section 4.1, sums to 1).
 * P, z, grad_z: device fp32 [n_rows, S], S = p->seq_len, row-major; entries
 * after t_i are never read. rows: device int32 [n_rows]; a row whose t_i is
 * outside [0, S) gets kl 0 and a zero gradient row. kl [n_rows] and loss [1]:
 * device fp32. kl, loss and grad_z may each be NULL, except that loss needs kl.
 * All buffers are caller-owned; the call is stream-ordered and allocates
 * nothing. Fields used: seq_len. n_rows = 0 is a no-op.
 */
int sp_kl_loss(const sp_problem *p, const int32_t *rows, int32_t n_rows, const float *P,
               const float *z, float *kl, float *loss, float *grad_z, hipStream_t stream);

/* Device workspace (bytes) an operation needs for problem p; 0 = none. */
int sp_workspace_bytes(const sp_problem *p, int op, size_t *bytes);

/* Static, human-readable text for a status code. */
const char *sp_status_string(int status);

/* SP_VERSION of the built library. */
int sp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPARSE_PREFILL_H_ */
