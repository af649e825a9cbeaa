/*
 * sevo.h — C ABI of libsevo.so: the population-batched decode step of
 * verifier-free evolution (Squeeze Evolve, arXiv 2604.07725) on one MI355X.
 *
 * What the library computes.  In each evolution loop the method hands every
 * group of K candidates to a model, which reads them as context and decodes one
 * refined candidate (method section, "Recombination" paragraph; Algorithm 1,
 * aggregation line).  The hot path is therefore one autoregressive decode step
 * for a whole population: N candidates, each with its own KV cache of ragged
 * length, advanced one token per step, returning the sampled token id and its
 * log-probability (the per-token log-probabilities the fitness signal of
 * Eq. 1 is built from; full-vocabulary sampling at temperature T as in the
 * generation hyper-parameter table).
 *
 * Conventions shared by every entry point
 *   - All tensors are caller-owned DEVICE memory unless a field says "host".
 *     The library never allocates on the hot path; scratch space comes from a
 *     caller-provided workspace sized by the matching *_workspace_bytes query.
 *     sevo_init_model allocates once (the RoPE table) and sevo_free_model
 *     releases it.
 *   - bf16 = IEEE binary32 with the low 16 bits dropped, stored as uint16.
 *   - Calls are stream-ordered and asynchronous: they enqueue kernels on
 *     `stream` (a hipStream_t; NULL = the legacy default stream) and return
 *     without synchronising.  Outputs are valid once the stream reaches them.
 *   - Every device pointer must be 16-byte aligned; row strides are in
 *     elements.
 *   - Errors: a non-zero sevo_status; outputs are then undefined.  No C++
 *     exception or abort crosses the ABI.  sevo_last_error() returns a
 *     thread-local message describing the most recent failure on the calling
 *     thread.  Host-visible scalars are validated on every call; the contents
 *     of device-resident page tables, lengths and positions are NOT validated
 *     on the hot path (sevo_validate_paging checks them on demand).
 *   - Paged KV cache, one KV pool per layer, page size 16:
 *       pool bf16 [num_pages][n_kv_heads][2][16 head_dim]: for each (page, kv
 *       head) the K tile, then the V tile (one contiguous 8 KB at head_dim 128)
 *       K tile: dims in blocks of 32, each block token-major: element (slot s,
 *               dim e) at ((e/32)*16 + s)*32 + e%32
 *       V tile: dim-major: element (s, e) at e*16 + s
 *     Logical key t of candidate i lives in physical page
 *     page_table[i * max_pages + t / 16], slot t % 16.  One page table serves
 *     all layers.  Physical page order is arbitrary (any permutation gives
 *     bit-identical results).
 *   - GQA: query head j reads KV head j / (n_q_heads / n_kv_heads).
 *   - GEMM operand layouts.  Both are built from the operand fragment of one
 *     16x16x32 bf16 matrix-core instruction: 16 rows x 32 columns stored as
 *     64 runs of 8 values, run index 16 ((c / 8) % 4) + r % 16, so a fragment
 *     is one contiguous 1 KB block.
 *       packed weight W [n_out][k] (n_out % 64 == 0, k % 32 == 0): element
 *         (r, c) at ((r/64 * k/32 + c/32) * 4 + (r/16) % 4) * 512
 *                   + (16 ((c/8) % 4) + r % 16) * 8 + c % 8
 *         (superblocks of 64 rows; per 32-column step the four 16-row
 *         fragments of a superblock are adjacent).  sevo_pack_weight builds it
 *         from row-major [n_out][k].
 *       tiled activation X [m][k] (k % 32 == 0): element (r, c) at
 *         (r/16 * k/32 + c/32) * 512 + (16 ((c/8) % 4) + r % 16) * 8 + c % 8,
 *         with m rounded up to a multiple of 16 rows (padding rows are never
 *         read into a stored result and need no initialisation).
 */
#ifndef SEVO_H
#define SEVO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t sevo_status;
#define SEVO_OK 0
#define SEVO_ERR_INVALID_ARGUMENT 1   /* null pointer, bad size, misalignment   */
#define SEVO_ERR_UNSUPPORTED 2        /* shape outside the supported set         */
#define SEVO_ERR_WORKSPACE_TOO_SMALL 3
#define SEVO_ERR_OUT_OF_MEMORY 4      /* only sevo_init_model allocates          */
#define SEVO_ERR_HIP 5                /* a HIP runtime call or launch failed     */
#define SEVO_ERR_BAD_PAGE_TABLE 6     /* sevo_validate_paging found a bad entry  */

#define SEVO_PAGE_SIZE 16

const char* sevo_status_string(sevo_status s);
/* Thread-local detail of the most recent failure on this thread ("" if none). */
const char* sevo_last_error(void);
/* Library version string, e.g. "sevo 0.1 gfx950". */
const char* sevo_version(void);

/* ------------------------------------------------------------------ model */

/* Decoder shape.  Supported: head_dim in {64, 128}; n_q_heads % n_kv_heads == 0
 * with n_q_heads / n_kv_heads in {1, 2, 4, 8}; page_size == 16; hidden, ffn and
 * n_q_heads * head_dim multiples of 128; vocab a multiple of 64; qk_norm in
 * {0, 1}; rms_eps > 0.
 * Mixture of experts (n_experts > 0; the FFN of every layer; ffn is then
 * unused): the Qwen3-MoE layer -- router logits h W_r^T, the n_experts_active
 * largest (ties to the lower expert index), weights = softmax over the
 * selected logits (the router probabilities of the selected experts,
 * renormalised), FFN(h) = sum over them of w_e * SwiGLU expert e.  Supported:
 * n_experts a multiple of 64 up to 256; 1 <= n_experts_active <= 16;
 * expert_ffn a multiple of 32. */
typedef struct {
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab;
  int32_t page_size;    /* must be 16 */
  int32_t max_position; /* RoPE table covers positions [0, max_position) */
  int32_t qk_norm;      /* 1: per-head RMSNorm of q and k before RoPE (Qwen3 style) */
  float rope_theta;     /* rotate-half RoPE base, e.g. 1e6 */
  float rms_eps;        /* RMSNorm epsilon, e.g. 1e-6 */
  int32_t n_experts;        /* 0 = dense SwiGLU FFN */
  int32_t n_experts_active; /* experts per token (top-k) */
  int32_t expert_ffn;       /* intermediate size of one expert */
} sevo_model_config;

/* Borrowed bf16 weight pointers (device); they must outlive the model.  The
 * per-layer members are HOST arrays of n_layers device pointers.  Shapes are
 * [out][in]; embed is row-major, the projection matrices are in the packed
 * weight layout (sevo_pack_weight, kind SEVO_PACK_PLAIN unless noted):
 *   embed [vocab][hidden] (row-major);  lm_head [vocab][hidden] (packed)
 *   final_norm, attn_norm, ffn_norm [hidden]
 *   w_qkv     [(n_q_heads + 2 n_kv_heads) head_dim][hidden]  rows: q, k, v
 *   q_norm, k_norm [head_dim]        (unused when qk_norm == 0; may be NULL)
 *   w_o       [hidden][n_q_heads head_dim]
 *   w_gate_up [2 ffn][hidden]        rows 0..ffn-1 gate, ffn..2ffn-1 up, packed
 *                                    with kind SEVO_PACK_GATE_UP
 *   w_down    [hidden][ffn]
 * A mixture-of-experts model (n_experts > 0) leaves w_gate_up / w_down NULL and
 * gives, per layer (Fe = expert_ffn, E = n_experts):
 *   w_router         [E][hidden] (packed)
 *   w_expert_gate_up [E][2 Fe][hidden]: expert e's matrix (gate rows, then up
 *                    rows) at element offset e * 2 Fe * hidden, each packed
 *                    with kind SEVO_PACK_GATE_UP
 *   w_expert_down    [E][hidden][Fe]: expert e at e * hidden * Fe, packed */
typedef struct {
  const void* embed;
  const void* lm_head;
  const void* final_norm;
  const void* const* attn_norm;
  const void* const* w_qkv;
  const void* const* q_norm;
  const void* const* k_norm;
  const void* const* w_o;
  const void* const* ffn_norm;
  const void* const* w_gate_up;
  const void* const* w_down;
  const void* const* w_router;
  const void* const* w_expert_gate_up;
  const void* const* w_expert_down;
} sevo_weights;

typedef struct sevo_model sevo_model;

/* Creates the model a population decodes with.  The paper serves its own
 * trained models and states no layer details; the decoder here is the pre-norm
 * GQA transformer of the Qwen3 family that the workloads are shaped after
 * (dense SwiGLU or mixture-of-experts FFN; the models of the System
 * Implementation subsection and the generation hyper-parameter table).
 * Validates the shape, copies the pointer tables and builds the RoPE cos/sin
 * table (angles in double, stored fp32) on the current device.
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, OUT_OF_MEMORY, HIP. */
sevo_status sevo_init_model(const sevo_model_config* cfg, const sevo_weights* w,
                            sevo_model** out);
void sevo_free_model(sevo_model* m);

/* ------------------------------------------------------------------ attention */

/* Paged GQA split-KV decode attention (one query token per candidate): the
 * attention of one decode step of LLM aggregation, where a candidate's context
 * is the K concatenated candidates of its group (Recombination paragraph of the
 * method section; Algorithm 1, aggregation line):
 *   o[i][j] = softmax_t(scale * q[i][j] . K_i[c][t]) V_i[c][t],  t < seq_lens[i],
 * c = j / (n_q_heads / n_kv_heads).  Each candidate's pages are cut into
 * splits of ceil(max_pages / S) logical pages, where S is num_splits raised as
 * needed so that a split spans at most 512 pages; every split yields an
 * online-softmax partial (running max, sum, weighted V) that a combine pass
 * merges in split order, so the result is deterministic.
 *   q        bf16 [n][n_q_heads][head_dim]
 *   kv_pool  paged layout above (bf16)
 *   page_table int32 [n][max_pages];  seq_lens int32 [n], 0 <= len <= 16 max_pages
 *   (a candidate with len 0 gets o = 0)
 *   out      bf16 [n][n_q_heads][head_dim]
 *   num_splits 0 = chosen by the library (see sevo_attn_plan_splits)
 * A page id outside [0, num_pages) contributes no keys (it is never read).
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, WORKSPACE_TOO_SMALL, HIP. */
typedef struct {
  int32_t n, n_q_heads, n_kv_heads, head_dim, page_size, max_pages, num_splits;
  int64_t num_pages; /* pages in each pool; ids outside [0, num_pages) are skipped */
  const void* q;
  const void* kv_pool;
  const int32_t* page_table;
  const int32_t* seq_lens;
  float scale;
  void* out;
  void* workspace;
  size_t workspace_bytes;
} sevo_attn_args;

sevo_status sevo_attn_decode(const sevo_attn_args* a, void* stream);

/* Separate K and V pools in the plain paged layout, bf16
 * [num_pages][n_kv_heads][16 slots][head_dim] each (slot-major rows), ->
 * the fused pool above (dst kv_pool, 2 x the bytes of one source pool), so a
 * caller that keeps the plain layout (for example one filled by another
 * prefill engine) can hand its cache to the attention and the decode step of
 * LLM aggregation (Recombination paragraph of the method section; Algorithm
 * 1, aggregation line).  Pure data movement: every element is copied bit for
 * bit.  head_dim 64 or 128 (else UNSUPPORTED); the three pools are
 * caller-owned, 16-byte aligned, and dst must not overlap either source
 * (INVALID_ARGUMENT).  num_pages 0 is a no-op.  Stream-ordered; not part of
 * the decode step. */
sevo_status sevo_pack_kv(const void* k_pool, const void* v_pool, int64_t num_pages,
                         int32_t n_kv_heads, int32_t head_dim, void* kv_pool, void* stream);
/* Split count the library uses when num_splits == 0. */
int32_t sevo_attn_plan_splits(int32_t n, int32_t n_kv_heads, int32_t max_pages);
/* Workspace for sevo_attn_decode with the given split count (0 = planned). */
size_t sevo_attn_workspace_bytes(int32_t n, int32_t n_q_heads, int32_t n_kv_heads,
                                 int32_t head_dim, int32_t max_pages, int32_t num_splits);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * attention as sevo_attn_decode, identical bits, with the split partials in a
 * fixed device array of the library instead of a caller workspace (the
 * workspace and workspace_bytes fields are ignored).  The array holds
 * SEVO_NOALLOC_SCRATCH_BYTES (32 MiB) on each GPU the library runs on, until
 * the process ends; a call whose partials need more
 * (n_q_heads * n * splits * (head_dim + 2) * 4 bytes, rounded to 256-byte
 * blocks) returns WORKSPACE_TOO_SMALL before launching anything.  Every call
 * on one GPU shares that GPU's array: calls that overlap in time on one GPU
 * (other streams, other threads) race and must be ordered by the caller.
 * The stream must belong to the current device.  Nothing here calls
 * hipMalloc or hipFree; the first call on a device looks up the array's
 * address (hipGetSymbolAddress), so make it outside any graph capture.
 * Errors: as sevo_attn_decode. */
#define SEVO_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
sevo_status sevo_attn_decode_noalloc(const sevo_attn_args* a, void* stream);

/* ------------------------------------------------------------------ prefill */

/* Causal GQA attention of a prefill: the forward pass the cross-model
 * confidence engine runs over a whole prompt + trajectory (the "Confidence
 * engine" paragraph of the System Implementation subsection; the prefill
 * engine appendix), for a batch of sequences back to back.  Token t of
 * sequence s sits at position pos(t) = start_pos[s] + (t - seq_starts[s]) and
 * attends to every key up to its own position:
 *   o[t][j] = softmax_{u <= pos(t)}(scale * q[t][j] . K_s[c][u]) V_s[c][u],
 * c = j / (n_q_heads / n_kv_heads), keys read from the paged pool through row
 * s of the page table.  The keys and values of positions 0..pos(t) must be in
 * the pool already (sevo_qk_norm_rope_append writes a prefill's own keys).
 *   q          bf16 [total_tokens][n_q_heads][head_dim]
 *   kv_pool    paged layout above (bf16)
 *   page_table int32 [n_seqs][max_pages]
 *   seq_starts int32 [n_seqs + 1] (device): non-decreasing token offsets,
 *              seq_starts[0] = 0, seq_starts[n_seqs] = total_tokens
 *   start_pos  int32 [n_seqs] (device) or NULL (every sequence starts at 0)
 *   out        bf16 [total_tokens][n_q_heads][head_dim]
 *   max_seq_len (host) >= every sequence length: sizes the grid (rows of a
 *              longer sequence past it are not computed); a value below the
 *              mean length total_tokens / n_seqs is rejected (INVALID_ARGUMENT)
 * The probabilities are rounded to bf16 for the P V product (fp32
 * accumulation; the softmax statistics stay fp32).  A page id outside
 * [0, num_pages) contributes no keys, as in sevo_attn_decode (it is never
 * read; a row that sees no key at all gets o = 0).
 * Device arrays are not validated.  Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP. */
typedef struct {
  int32_t n_seqs, total_tokens, max_seq_len;
  int32_t n_q_heads, n_kv_heads, head_dim, page_size, max_pages;
  int64_t num_pages;
  const void* q;
  const void* kv_pool;
  const int32_t* page_table;
  const int32_t* seq_starts;
  const int32_t* start_pos;
  float scale;
  void* out;
} sevo_prefill_attn_args;

sevo_status sevo_attn_prefill(const sevo_prefill_attn_args* a, void* stream);

/* The cross-model confidence engine: one prefill-only forward pass of the
 * scoring model over every sequence of a batch (prompt + trajectory), reduced
 * on the device to one confidence per sequence (Eq. 1 per position, Eq. 2's
 * C(tau) per sequence; the "Confidence engine" paragraph of the System
 * Implementation subsection and the prefill engine appendix).  Per layer the
 * steps of sevo_decode_step run for all total_tokens tokens at once, with the
 * causal prefill attention of sevo_attn_prefill; the keys and values of every
 * token are written into the pools (a KV cache a decode can continue from).
 * A mixture-of-experts model runs its expert FFN on chunks of moe_chunk
 * tokens (rounded up to 16; 0 or more than 65536 = 65536; lowered, to a
 * multiple of 16, as needed to keep chunk * max(hidden, n_experts_active *
 * expert_ffn) * 2 below 2^31 bytes): routing, expert lists and the per-slot
 * outputs of a chunk live in the workspace, and each token's k expert outputs
 * are summed in slot order.
 * Then, for each scored row r -- a packed token index whose next-token
 * distribution is scored --
 *   c_r = logsumexp(logits_r) - mean of the conf_topk largest logits_r
 * with logits_r = RMSNorm(x_r) g_final W_lm^T (fp32, T = 1), and
 *   out_conf[s] = mean of c_r over the scored rows inside sequence s
 *                 (C(tau) of Eq. 2; 0 for a sequence without scored rows).
 * Only the scored rows go through the LM head (in chunks of 4096 rows).
 *   tokens      int32 [total_tokens], sequences back to back
 *   seq_starts  int32 [n_seqs + 1] (device), start_pos int32 [n_seqs] (device)
 *               or NULL: as in sevo_attn_prefill; positions must be below the
 *               model's max_position
 *   page_table  int32 [n_seqs][max_pages]: pages for every key position
 *   kv_pools    HOST array of n_layers pool pointers; a caller that does not
 *               keep the cache may pass one pool for every layer (a layer's
 *               keys are only read inside that layer)
 *   max_seq_len host bound of the sequence lengths (at least the mean length
 *               total_tokens / n_seqs, else INVALID_ARGUMENT)
 *   conf_topk   K_l of Eq. 1, 1..32
 *   scored_rows int32 [n_scored] (device): strictly increasing packed token
 *               indices (not validated on the device)
 *   out_conf    fp32 [n_seqs];  out_row_conf fp32 [n_scored] or NULL
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, WORKSPACE_TOO_SMALL, HIP. */
typedef struct {
  int32_t n_seqs, total_tokens, max_seq_len;
  const int32_t* tokens;
  const int32_t* seq_starts;
  const int32_t* start_pos;
  const int32_t* page_table;
  int32_t max_pages;
  int64_t num_pages;
  void* const* kv_pools;
  int32_t conf_topk;
  int32_t n_scored;
  const int32_t* scored_rows;
  float* out_conf;
  float* out_row_conf;
  void* workspace;
  size_t workspace_bytes;
  int32_t moe_chunk;  /* MoE models: tokens per expert-FFN chunk, 0 = 65536 (the
                         largest; sevo_prefill_workspace_bytes sizes for it);
                         negative: INVALID_ARGUMENT */
} sevo_prefill_args;

sevo_status sevo_prefill_confidence(sevo_model* m, const sevo_prefill_args* a, void* stream);
size_t sevo_prefill_workspace_bytes(const sevo_model* m, int32_t total_tokens, int32_t n_scored);

/* ------------------------------------------------------------------ sampling */

/* Full-vocabulary log-softmax and Gumbel-max sample, per candidate i:
 *   z = logits[i] / T;  id = argmax_v (z_v + G_v)  (ties -> lowest v);
 *   logprob = z_id - logsumexp(z).
 * G_v = -log(-log u_v), u_v = ((w >> 9) + 0.5) 2^-23 with w the (v & 3)-th
 * word of Philox4x32-10 (Salmon et al., SC'11) on counter
 * (v >> 2, position_i, uid_i lo, uid_i hi) and key (seed lo, seed hi).  Noise
 * is keyed by candidate uid and position, never by call count, so a resumed or
 * re-ordered population draws the same tokens.  T == 0: greedy argmax, logprob
 * under T = 1.  T < 0 or non-finite: INVALID_ARGUMENT.  A row with no
 * comparable perturbed value (every logit NaN) gets id -1 and logprob NaN.
 *   logits fp32 [n][ld] (first vocab entries used); cand_uid uint64 [n];
 *   positions int32 [n];  out_tokens int32 [n];  out_logprobs fp32 [n].
 * Truncated sampling (the top-k / top-p / min-p rows of the generation
 * hyper-parameter table), active when top_k > 0 (1..32, at most vocab):
 *   kept = the top_k logits in (value desc, index asc) order -- temperature
 *   does not change the set; with z = logit / T over it, min-p keeps
 *   z_j >= z_0 + log(min_p) (min_p in [0, 1], 0 = off), then top-p keeps, in
 *   that order, each entry whose preceding cumulative probability
 *   (renormalised over the min-p set) is below top_p (top_p in (0, 1], 1 = off);
 *   id = argmax over kept of (z_v + G_v) with the noise above;
 *   logprob = z_id - logsumexp(kept z), the distribution that is sampled.
 *   T == 0: the first entry; truncation and logprob evaluated at T = 1.
 *   top_k == 0 needs top_p == 1 and min_p == 0 (UNSUPPORTED otherwise).
 * Self-confidence (the group-confidence fitness signal, Eq. 1), computed in
 * the same passes when conf_topk > 0 (1..32, and at most vocab):
 *   c_i = -(1/K) * sum of the K largest log_softmax(logits[i]) entries
 *       = logsumexp(logits[i]) - mean of the K largest logits[i],
 * under the model's own distribution (T = 1) whatever the sampling T.
 *   out_conf fp32 [n] (nullable) receives c_i; conf_sum fp32 [n] (nullable) gets
 *   c_i added (a running sum over a trajectory's tokens: C = conf_sum / tokens).
 * Errors: INVALID_ARGUMENT, UNSUPPORTED (max(top_k, conf_topk) * ceil(vocab /
 * 4096) > 6144; top_p / min_p without top_k), WORKSPACE_TOO_SMALL, HIP. */
typedef struct {
  const float* logits;
  int32_t n, vocab;
  int64_t ld;
  float temperature;
  uint64_t seed;
  const uint64_t* cand_uid;
  const int32_t* positions;
  int32_t* out_tokens;
  float* out_logprobs;
  int32_t top_k;     /* 0 = full vocabulary */
  float top_p;       /* 1 = off */
  float min_p;       /* 0 = off */
  int32_t conf_topk; /* 0 = no confidence */
  float* out_conf;
  float* conf_sum;
  void* workspace;
  size_t workspace_bytes;
} sevo_sample_args;

sevo_status sevo_logprob_sample(const sevo_sample_args* a, void* stream);
size_t sevo_sample_workspace_bytes(int32_t n, int32_t vocab);

/* Group confidence of Eq. 2 from the per-candidate running sums:
 *   GC[g] = (1/K) sum_{k<K} conf_sum[c] / token_counts[c],  c = groups[g*K + k]
 * (C(tau) = conf_sum / token count is the candidate confidence).
 *   conf_sum fp32 [n];  token_counts int32 [n] (> 0 for every grouped
 *   candidate);  groups int32 [n_groups][group_size];  out_gc fp32 [n_groups].
 * Candidate indices are not validated on the device.
 * Errors: INVALID_ARGUMENT, HIP. */
sevo_status sevo_group_confidence(const float* conf_sum, const int32_t* token_counts,
                                  const int32_t* groups, int32_t n_groups, int32_t group_size,
                                  float* out_gc, void* stream);

/* ------------------------------------------------------------------ decode step */

/* One decode step of the whole population through the model (the step that
 * LLM aggregation repeats for every candidate: the Recombination paragraph of
 * the method section and Algorithm 1's aggregation line; the returned
 * log-probabilities are the per-token terms of Eq. 1):
 *   x = embed[token];  per layer: h = RMSNorm(x) g_attn;  [q|k|v] = h W_qkv^T;
 *   (qk_norm) q, k <- per-head RMSNorm * g_q / g_k;  RoPE(q, k) at p_i;
 *   append k, v as key number p_i;  o = attention over keys 0..p_i;
 *   x += o W_o^T;  h = RMSNorm(x) g_ffn;  x += (silu(h W_g^T) * (h W_u^T)) W_d^T;
 * then logits = RMSNorm(x) g_final W_lm^T (fp32) and the sampler above.
 * Storage: residual x fp32; GEMM inputs, q, K/V, attention output and the
 * SwiGLU product bf16; logits fp32.
 *   tokens int32 [n];  positions int32 [n] (p_i = keys cached before the step;
 *   the caller must have a page for slot p_i, and p_i < max_position);
 *   page_table int32 [n][max_pages];  kv_pools: HOST array of
 *   n_layers device pool pointers;  cand_uid uint64 [n];
 *   out_tokens int32 [n];  out_logprobs fp32 [n];
 *   out_logits fp32 [n][vocab] or NULL (then kept in the workspace);
 *   top_k, top_p, min_p: truncated sampling; conf_topk, out_conf, conf_sum:
 *   the sampler's self-confidence (both above);
 *   out_hidden fp32 [n_layers + 1][n][hidden] or NULL: the residual stream x
 *   entering each layer (entry l) and after the last layer (entry n_layers),
 *   for layer-by-layer verification; one device-to-device copy per entry.
 * The library never changes positions or page tables: the caller advances p_i
 * and allocates pages.  Errors: INVALID_ARGUMENT, UNSUPPORTED,
 * WORKSPACE_TOO_SMALL, HIP. */
typedef struct {
  int32_t n;
  const int32_t* tokens;
  const int32_t* positions;
  const int32_t* page_table;
  int32_t max_pages;
  int64_t num_pages; /* pages in each pool (bounds every page access) */
  void* const* kv_pools;
  const uint64_t* cand_uid;
  uint64_t seed;
  float temperature;
  int32_t num_splits;
  int32_t* out_tokens;
  float* out_logprobs;
  float* out_logits;
  int32_t top_k;
  float top_p;
  float min_p;
  int32_t conf_topk;
  float* out_conf;
  float* conf_sum;
  void* workspace;
  size_t workspace_bytes;
  float* out_hidden; /* nullable, see above */
} sevo_step_args;

sevo_status sevo_decode_step(sevo_model* m, const sevo_step_args* a, void* stream);
size_t sevo_step_workspace_bytes(const sevo_model* m, int32_t n, int32_t max_pages,
                                 int32_t num_splits);

/* ------------------------------------------------------------------ sub-steps
 * The steps of sevo_decode_step, exposed one by one so each can be checked
 * and timed on its own.  Same conventions as above. */

/* x[i][:] = embed[tokens[i]][:] as fp32.  embed bf16 [vocab][hidden]; hidden % 8 == 0.
 * A token id outside [0, vocab) gives a zero row (the table is never read out of range). */
sevo_status sevo_embed(const void* embed, const int32_t* tokens, int32_t n, int32_t hidden,
                       int32_t vocab, float* x, void* stream);

/* out[r][:] = bf16(x[r][:] / sqrt(mean(x[r]^2) + eps) * gain), x fp32 [rows][cols],
 * gain bf16 [cols].  cols % 4 == 0. */
sevo_status sevo_rmsnorm(const float* x, const void* gain, int32_t rows, int32_t cols,
                         float eps, void* out, void* stream);

/* The residual update + RMSNorm that joins the sub-layers of a decoder layer:
 *   x[r][:] += sum over s < n_partials of partials[s][r][:]   (in s order,
 *              written back to x; x unchanged when n_partials = 0)
 *   out[r][:] = bf16(x[r][:] / sqrt(mean(x[r]^2) + eps) * gain)
 * x fp32 [rows][cols]; partials fp32 [n_partials][rows][cols] (the split-K
 * partials of the projection before it; NULL when n_partials = 0); gain bf16
 * [cols]; out bf16 in the tiled activation layout the projections read
 * (16-row tiles, a buffer of ceil(rows / 16) * 16 rows; padding rows are not
 * written).  cols % 4 == 0, 0 <= n_partials <= 16.  Errors: INVALID_ARGUMENT. */
sevo_status sevo_add_rmsnorm(float* x, const float* partials, int32_t n_partials,
                             const void* gain, int32_t rows, int32_t cols, float eps, void* out,
                             void* stream);

/* Y = X W^T with X bf16 [m][k], W bf16 [n_out][k] in the packed weight layout
 * (for SWIGLU packed with kind SEVO_PACK_GATE_UP), fp32 accumulation on the
 * matrix cores, then the epilogue:
 *   SEVO_LINEAR_STORE  out fp32 [m][n_out]  = Y
 *   SEVO_LINEAR_ADD    out fp32 [m][n_out] += Y          (residual update)
 *   SEVO_LINEAR_SWIGLU out bf16 [m][n_out/2] = silu(Y[:, :n_out/2]) * Y[:, n_out/2:]
 * flags: SEVO_LINEAR_X_TILED     X in the tiled activation layout (ldx unused;
 *                                else row-major with row stride ldx, ldx % 8 == 0)
 *        SEVO_LINEAR_OUT_TILED   SWIGLU output in the tiled activation layout
 * k % 32 == 0; n_out % 64 == 0.  k_splits 0 = chosen by the library (SWIGLU
 * always uses one split). */
#define SEVO_LINEAR_STORE 0
#define SEVO_LINEAR_ADD 1
#define SEVO_LINEAR_SWIGLU 2
#define SEVO_LINEAR_X_TILED 1
#define SEVO_LINEAR_OUT_TILED 2
typedef struct {
  int32_t m, n_out, k, ldx, mode, k_splits, flags;
  const void* x;
  const void* w;
  void* out;
  void* workspace;
  size_t workspace_bytes;
} sevo_linear_args;

sevo_status sevo_linear(const sevo_linear_args* a, void* stream);
size_t sevo_linear_workspace_bytes(int32_t m, int32_t n_out, int32_t k, int32_t k_splits);
/* The plan of the skinny kernel that sevo_linear runs for m < 256 (and the
 * decode step for its projections): plan[0] = K splits, plan[1] = k per split,
 * plan[2] = 16-row weight blocks per workgroup (for SWIGLU gate and up blocks,
 * an even count).  The planner aims at one round of 256 equal workgroups (one
 * per CU).  Writes plan[0..2] (caller-owned host memory) and returns SEVO_OK;
 * INVALID_ARGUMENT for a null plan or a shape outside m in [1, 255],
 * n_out % 64 == 0, k % 32 == 0, mode in {STORE, ADD, SWIGLU}. */
sevo_status sevo_linear_plan(int32_t m, int32_t n_out, int32_t k, int32_t k_splits, int32_t mode,
                             int32_t* plan);

/* Row-major bf16 [n_out][k] (src) -> packed weight layout (dst, a separate
 * buffer of the same size).  SEVO_PACK_GATE_UP treats rows 0..n_out/2-1 as
 * gate rows and the rest as up rows and puts gate rows 32 s..32 s+31 and up
 * rows n_out/2 + 32 s.. in superblock s (logical order gate, then up), the form
 * the SWIGLU epilogue reads.  n_out % 64 == 0, k % 32 == 0.  A one-time
 * preparation of model weights, not part of the decode step. */
#define SEVO_PACK_PLAIN 0
#define SEVO_PACK_GATE_UP 1
sevo_status sevo_pack_weight(const void* src, void* dst, int32_t n_out, int32_t k, int32_t kind,
                             void* stream);

/* The fused QK-RMSNorm + RoPE + KV append of one layer.
 *   qkv fp32 [n][(n_q_heads + 2 n_kv_heads) head_dim] (the QKV projection)
 *   q_out bf16 [n][n_q_heads][head_dim]: RoPE(RMSNorm(q) g_q) at p_i
 *   kv_pool: slot p_i of every candidate receives RoPE(RMSNorm(k) g_k) (K tile) and v (V tile).
 * Uses the model's RoPE table, norm gains and shape (layer selects the gains). */
sevo_status sevo_qk_norm_rope_append(const sevo_model* m, int32_t layer, const float* qkv,
                                     int32_t n, const int32_t* positions,
                                     const int32_t* page_table, int32_t max_pages,
                                     int64_t num_pages, void* q_out, void* kv_pool,
                                     void* stream);

/* The mixture-of-experts FFN of one layer on normed inputs (the sub-step of a
 * MoE decode step): h bf16 in the tiled activation layout, n rows (a buffer
 * of ceil(n / 16) * 16 rows; padding rows are not read), device memory owned
 * by the caller like every output.
 *   out_experts int32 [n][k] (selected experts, largest logit first; always k
 *   distinct experts, also when logits are not finite);
 *   out_weights fp32 [n][k]; out_partials fp32 [k][n][hidden]:
 *   partial j of token t = w_{t,j} * SwiGLU expert out_experts[t][j] (h_t), so
 *   FFN(h_t) = the sum of the k partials in slot order.
 * n k <= 2^30.  Errors: INVALID_ARGUMENT, UNSUPPORTED (dense model),
 * WORKSPACE_TOO_SMALL, HIP. */
sevo_status sevo_moe_ffn(const sevo_model* m, int32_t layer, const void* h, int32_t n,
                         int32_t* out_experts, float* out_weights, float* out_partials,
                         void* workspace, size_t workspace_bytes, void* stream);
size_t sevo_moe_workspace_bytes(const sevo_model* m, int32_t n);

/* ------------------------------------------------------------------ utilities */

/* Streaming-read microbenchmark (measurement tooling, not part of the decode
 * step): the measured HBM read ceiling the decode attention is compared with,
 * next to the 8 TB/s specification.  Reads `bytes` of device memory at buf
 * (16-byte aligned) once:
 *   page_order NULL: a grid-stride sequential read of bytes / 16 16-byte words;
 *   else whole 8 KB pages in the order page_order [bytes / 8192] (int32 page
 *   indexes; an index outside [0, bytes / 8192) is skipped), one wave per page,
 *   the decode attention's access pattern.
 * grid = workgroups (256 threads), 1..2^20; sink receives one 16-byte word
 * per workgroup (device memory of >= 16 * grid bytes, caller-owned).  Time it
 * with events on `stream`.  Errors: INVALID_ARGUMENT, HIP. */
sevo_status sevo_hbm_read_probe(const void* buf, size_t bytes, const int32_t* page_order,
                                int32_t grid, void* sink, void* stream);

/* Synthetic-input generator (device twin of the host generator): element e of
 * dst (e < count) = bf16_rne(fp32(s - 131070) * mul [+ add]) with s the sum of
 * the four 16-bit fields of SplitMix64(key + (offset + e + 1) 0x9E3779B97F4A7C15).
 * Pure input generation, not part of the decode step. */
sevo_status sevo_fill_normal_bf16(void* dst, int64_t count, uint64_t key, int64_t offset,
                                  float mul, float add, int32_t use_add, void* stream);

/* Copies page_table / lengths to the host and checks that every logical page
 * a candidate needs (ceil(len_i / 16) pages) is in [0, num_pages) and that no
 * physical page is used twice.  Synchronises the stream.  Returns
 * SEVO_ERR_BAD_PAGE_TABLE with a message on the first violation. */
sevo_status sevo_validate_paging(const int32_t* page_table, const int32_t* lengths, int32_t n,
                                 int32_t max_pages, int64_t num_pages, void* stream);

/* ------------------------------------------------------------------ timing
 * Measurement aid: while a recording is open, the launches of the selected
 * kinds (inside sevo_decode_step and sevo_prefill_confidence; the attention
 * kinds also in sevo_attn_decode and sevo_attn_prefill) are bracketed by HIP
 * events on the stream they run on.  Process-wide; launches beyond max_launches are not timed; one recording at a
 * time.  kinds is a mask of (1u << SEVO_PROF_*).  sevo_profile_end waits for
 * the recorded events and returns, per kind, the summed milliseconds and the
 * number of timed launches (arrays of SEVO_PROF_NUM_KINDS entries; either may
 * be NULL).  Recording adds two event records per timed launch. */
#define SEVO_PROF_ATTN_SPLIT 0    /* split-KV attention kernel           */
#define SEVO_PROF_ATTN_COMBINE 1  /* cross-split combine                 */
#define SEVO_PROF_QKV 2           /* QKV projection                      */
#define SEVO_PROF_ATTN_OUT 3      /* output projection                   */
#define SEVO_PROF_GATE_UP 4       /* gate/up projection + SwiGLU         */
#define SEVO_PROF_DOWN 5          /* down projection                     */
#define SEVO_PROF_LM_HEAD 6       /* LM head                             */
#define SEVO_PROF_NORM 7          /* residual add + RMSNorm              */
#define SEVO_PROF_ROPE_APPEND 8   /* QK-norm + RoPE + KV append          */
#define SEVO_PROF_SAMPLE 9        /* log-softmax + Gumbel-max (+ confidence) */
#define SEVO_PROF_EMBED 10        /* embedding gather                    */
#define SEVO_PROF_ATTN_PREFILL 11 /* causal prefill attention            */
#define SEVO_PROF_MOE_ROUTE 12    /* MoE router GEMM, top-k, expert lists */
#define SEVO_PROF_MOE_EXPERTS 13  /* MoE expert gate/up + down GEMMs      */
#define SEVO_PROF_NUM_KINDS 14
sevo_status sevo_profile_begin(int32_t max_launches, uint32_t kinds);
sevo_status sevo_profile_end(float* total_ms, int32_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* SEVO_H */
