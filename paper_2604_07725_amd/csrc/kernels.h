// Internal launchers of libsevo (C++ linkage, not part of the ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sevo {

typedef uint16_t bf16_t;

// ---- norm_rope.hip
hipError_t launch_embed(const bf16_t* embed, const int32_t* tokens, int n, int hidden,
                        int vocab, float* x, hipStream_t st);
hipError_t launch_rmsnorm(const float* x, const bf16_t* gain, int rows, int cols, float eps,
                          bf16_t* out, hipStream_t st);
// x += sum_s part[s] (split order; S == 0: nothing to add), then
// out = bf16(RMSNorm(x) * gain) in the tiled activation layout (the GEMM
// input).  part is [S][rows][cols] fp32.
// row_idx (optional): output row r takes source row row_idx[r] of x and of
// the partials (which then have part_rows rows); x is not written back.
hipError_t launch_add_rmsnorm(float* x, const float* part, int S, const bf16_t* gain, int rows,
                              int cols, float eps, bf16_t* out_tiled, hipStream_t st,
                              const int32_t* row_idx = nullptr, int part_rows = 0);
// per packed prefill token: page-table row (its sequence) and position
hipError_t launch_prefill_index(const int32_t* seq_starts, const int32_t* start_pos, int n_seqs,
                                int T, int32_t* row, int32_t* pos, hipStream_t st);
struct RopeAppendArgs {
  const float* qkv;  // [qkv_splits][n][(hq + 2 hkv) d]: summed in split order
  int qkv_splits;
  int n, hq, hkv, d;
  const int32_t* positions;
  const int32_t* page_table;
  int max_pages;
  int64_t num_pages;
  const float* rope_cos;  // [max_pos][d/2]
  const float* rope_sin;
  int max_pos;
  const bf16_t* q_gain;   // null when qk_norm == 0
  const bf16_t* k_gain;
  int qk_norm;
  float eps;
  bf16_t* q_out;
  bf16_t* kv_pool;  // [num_pages][hkv][2][16 d]: K tile, then V tile
  // page-table row of token i (null: row i); a prefill's tokens share the row
  // of their sequence
  const int32_t* row_of_token = nullptr;
};
hipError_t launch_qk_norm_rope_append(const RopeAppendArgs& a, hipStream_t st);
// separate K, V pools [tiles][16][d] -> the fused pool [tiles][2][16 d]; d 64 or 128
hipError_t launch_pack_kv(const bf16_t* k_src, const bf16_t* v_src, size_t tiles, int d,
                          bf16_t* kv, hipStream_t st);
hipError_t launch_fill_bf16(bf16_t* dst, int64_t count, uint64_t key, int64_t offset, float mul,
                            float add, int use_add, hipStream_t st);

// ---- attn_decode.hip
struct AttnArgs {
  int n, hq, hkv, d, max_pages, num_splits, chunk;
  int64_t num_pages;
  const bf16_t* q;
  const bf16_t* kv_pool;
  const int32_t* page_table;
  const int32_t* seq_lens;  // keys per candidate = seq_lens[i] + len_add
  int len_add;
  float scale;
  bf16_t* out;
  int out_tiled = 0;  // 1: out in the tiled activation layout of [n][hq d]
  float* part_ml;   // [n][hq][S][2]
  float* part_acc;  // [n][hq][S][d]
  // optional timing: recorded before the split kernel, between the two
  // kernels and after the combine (all null = no recording)
  hipEvent_t ev_begin = nullptr, ev_mid = nullptr, ev_end = nullptr;
};
hipError_t launch_attn_decode(const AttnArgs& a, hipStream_t st);

// ---- attn_prefill.hip: causal GQA attention of a prefill over the paged KV
// cache (the keys of every sequence's tokens already appended)
struct PrefillAttnArgs {
  int n_seqs, hq, hkv, d, max_pages, max_seq_len;
  int64_t num_pages;
  const bf16_t* q;            // [T][hq][d], sequences back to back
  const bf16_t* kv_pool;
  const int32_t* page_table;  // [n_seqs][max_pages]
  const int32_t* seq_starts;  // [n_seqs + 1] token offsets
  const int32_t* start_pos;   // [n_seqs] position of each sequence's first token (null: 0)
  float scale;
  bf16_t* out;                // row-major [T][hq][d], or tiled [T][hq d] when out_tiled
  int out_tiled;
  int total_tokens;           // T (the tiled layout's row count)
};
hipError_t launch_attn_prefill(const PrefillAttnArgs& a, hipStream_t st);

// ---- moe.hip: mixture-of-experts FFN of a decode step
constexpr int kMoeGroupRows = 256;  // rows per tile of the grouped large-M GEMM

struct MoeExpertArgs {
  int n, hidden, ffn, n_experts, top_k;
  const bf16_t* x;          // normed input, tiled [n][hidden]
  const bf16_t* w_gate_up;  // [E][2 ffn][hidden], each expert packed (gate/up superblocks)
  const bf16_t* w_down;     // [E][hidden][ffn], each expert packed
  const int32_t* offsets;   // [E + 1] assignment offsets per expert
  const int32_t* assign;    // [n k] assignments t * k + slot, expert-major
  const float* weights;     // [n k] routing weights
  bf16_t* act;              // [n k][ffn] SwiGLU products, row = assignment position
  float* part;              // [k][n][hidden] weighted expert outputs per slot
};
bool moe_supported(int n_experts, int top_k, int expert_ffn, int hidden);
// logits = sum of S split partials [S][n][E]; sel / w [n][k]
hipError_t launch_moe_route(const float* part, int S, int n, int E, int k, int32_t* sel,
                            float* w, hipStream_t st);
// out [n][H] = sum of the k slot partials [k][n][H] in slot order
hipError_t launch_moe_sum_slots(const float* part, int k, int n, int H, float* out,
                                hipStream_t st);
// offsets [E + 1], assign [nk] (entries expert-major, token order); with
// tile_off [E + 1]: each expert's first 256-entry tile (grouped GEMM)
// scratch (optional, moe_plan_scratch_bytes): from 4097 entries the plan runs
// as three launches over 1024-entry chunks instead of one workgroup
hipError_t launch_moe_plan(const int32_t* sel, int nk, int E, int32_t* offsets, int32_t* assign,
                           hipStream_t st, int32_t* tile_off = nullptr, int32_t* scratch = nullptr);
size_t moe_plan_scratch_bytes(int nk, int E);
// gate/up + SwiGLU into act, then down into part
hipError_t launch_moe_experts(const MoeExpertArgs& a, hipStream_t st);

// ---- linear.hip
struct LinearPlan {
  int k_splits;
  int k_chunk;
  int rb = 4;  // 16-row weight blocks per workgroup (SwiGLU: gate + up blocks)
};
LinearPlan plan_linear(int m, int n_out, int k, int k_splits, int mode);
size_t linear_workspace_bytes(int m, int n_out, int k, int k_splits, int mode);
// X operand: row-major with row stride ldx (x_tiled == 0) or the tiled
// activation layout; W: the packed weight layout (gate/up interleaved for SWIGLU).
// complete Y = X W^T with the STORE / ADD / SWIGLU epilogue (SWIGLU output
// bf16, row-major or tiled per out_tiled)
hipError_t launch_linear(int m, int n_out, int k, int ldx, int x_tiled, int mode,
                         const LinearPlan& plan, const bf16_t* x, const bf16_t* w, void* out,
                         int out_tiled, float* workspace, hipStream_t st);
// raw fp32 split partials out[split][m][n] (k_splits == 1: the product itself,
// added to out when accumulate)
hipError_t launch_linear_partials(int m, int n_out, int k, int ldx, int x_tiled,
                                  const LinearPlan& plan, const bf16_t* x, const bf16_t* w,
                                  float* out, int accumulate, hipStream_t st);
// ---- gemm_large.hip: one-pass Y = X W^T for large M (prefill token counts),
// same operand layouts and epilogue modes as launch_linear (no workspace)
constexpr int kLargeGemmMinM = 256;
bool gemm_large_supported(int m, int n_out, int k);
// grouped form (mixture of experts): m-tiles are 256-entry tiles of the
// experts' entry lists; the expert's weights at w + e n_out k
struct GroupArgs {
  const int32_t* offsets = nullptr;   // [E + 1] entry offsets
  const int32_t* assign = nullptr;    // [n k] entries t * k + slot
  const int32_t* tile_off = nullptr;  // [E + 1] first tile of each expert
  const float* weights = nullptr;     // [n k] routing weights (down)
  int E = 0, k = 1, n = 0;            // experts, top-k, tokens
};
// down 0: gate/up of every entry, x = the tiled normed input (m = tokens),
//   out bf16 act [n k][n_out / 2] at the entry positions (SwiGLU);
// down 1: x = act [n k][k] row-major (m = n k entries), out fp32
//   [k slots][n][n_out] = weight * product.  max_tiles_m >= sum of the
//   experts' tile counts (n k / 256 + E).
hipError_t launch_gemm_grouped(int down, int m, int n_out, int k, const bf16_t* x,
                               const bf16_t* w, void* out, const GroupArgs& g, int max_tiles_m,
                               hipStream_t st);
hipError_t launch_gemm_large(int m, int n_out, int k, int ldx, int x_tiled, int mode,
                             const bf16_t* x, const bf16_t* w, void* out, int out_tiled,
                             hipStream_t st);
// row-major [n_out][k] -> packed weight layout; gate_up: rows 0..n_out/2-1 are
// gate rows and the rest up rows, interleaved per superblock (32 + 32)
hipError_t launch_pack_weight(const bf16_t* src, bf16_t* dst, int n_out, int k, int gate_up,
                              hipStream_t st);

// ---- sample.hip
constexpr int kSampleChunk = 4096;  // vocab entries per partial workgroup
size_t sample_workspace_bytes(int n, int vocab);
// conf_k > 0: also the per-token confidence (written to out_conf and/or added
// to conf_sum, either may be null).  top_k > 0: truncated sampling (top-k, then
// min-p and top-p inside the top-k set).
hipError_t launch_logprob_sample(const float* logits, int n, int vocab, int64_t ld, float temp,
                                 uint64_t seed, const uint64_t* uid, const int32_t* positions,
                                 int32_t* out_tokens, float* out_lp, float* workspace,
                                 int conf_k, float* out_conf, float* conf_sum, hipStream_t st,
                                 int top_k = 0, float top_p = 1.f, float min_p = 0.f);
// a top-k / confidence list of list_len entries fits the chunk merge
bool sample_conf_supported(int vocab, int list_len);
// C of each sequence: the mean, in row order, of row_conf over the scored rows
// (strictly increasing packed token indices) inside [seq_starts[s],
// seq_starts[s + 1]); 0 for a sequence with none.
// streaming-read microbenchmark (measurement tooling, not the decode path)
hipError_t launch_hbm_read_probe(const void* buf, size_t bytes, const int32_t* page_order,
                                 int grid, void* sink, hipStream_t st);
hipError_t launch_seq_confidence(const float* row_conf, const int32_t* scored_rows, int n_scored,
                                 const int32_t* seq_starts, int n_seqs, float* out,
                                 hipStream_t st);
hipError_t launch_group_confidence(const float* conf_sum, const int32_t* counts,
                                   const int32_t* groups, int n_groups, int K, float* out,
                                   hipStream_t st);

}  // namespace sevo
