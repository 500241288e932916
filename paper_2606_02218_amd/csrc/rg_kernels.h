// Host-side launchers of the rollout kernels.  Every launcher enqueues on
// `st` and returns the launch status.  Row counts that change during decoding
// are read by the kernels from device memory (`d_rows`); the grids are sized
// by a host upper bound `rows_ub` and surplus blocks exit at once.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rg_device.h"

struct KvGeom {
  int page_tok;         // tokens per page (16)
  int n_layers, n_kv, head_dim;
  int64_t slab_elems;   // elements of one page in one layer: 2 * n_kv * page_tok * head_dim
  int64_t page_stride;  // elements from page p to page p + 1 within a layer
  int64_t layer_stride; // elements from layer l to layer l + 1 within a page
};

// Layer l of page p holds a key slab per kv head h at
//   p*page_stride + l*layer_stride + h*16*head_dim
// and a value slab at
//   p*page_stride + l*layer_stride + (n_kv + h)*16*head_dim.
// The pool is layer-major (page_stride = slab_elems, layer_stride =
// pool_pages * slab_elems): one layer's pages are contiguous, so a layer's
// attention pass touches 1/n_layers of the pool's address range.
// Both slabs are made of 16-byte granules of 8 elements (bf16): keys as
// [d/8][slot][8] (8 consecutive dims of one token), values as [slot/8][d][8]
// (8 consecutive tokens of one dim).  A quarter-wave of lanes reading the
// same dims of 4 neighbouring tokens (keys) or the same tokens of 4
// neighbouring dims (values) then touches 64 contiguous bytes.
__host__ __device__ inline int64_t kv_k_off(int slot, int d) { return (int64_t)(d >> 3) * 128 + slot * 8 + (d & 7); }
__host__ __device__ inline int64_t kv_v_off(int slot, int d, int hd) {
  return (int64_t)(slot >> 3) * hd * 8 + (int64_t)d * 8 + (slot & 7);
}

// Kernel timing hook.  The profiler arms a (start, stop) event pair for the
// next launch; a launcher that supports it takes the pair and launches its
// kernel with hipExtLaunchKernelGGL, so that the events time the kernel's own
// dispatch rather than the stream around it.
void rg_arm_launch_events(hipEvent_t start, hipEvent_t stop);
bool rg_take_launch_events(hipEvent_t* start, hipEvent_t* stop);   // disarms
bool rg_launch_events_armed();

// dtype: 0 = fp32 storage, 1 = bf16 storage.  Activation operands (`act`,
// `a_plane`) follow ActOut in rg_device.h: fp32 for fp32 models, hi/lo bf16
// planes a_plane elements apart for bf16 models.

// Output tile rows / columns launch_gemm uses for a row bound and width N.
int gemm_tile_rows(int dtype, int rows_ub, int N);
int gemm_tile_cols(int dtype, int rows_ub, int N, int K);

// Largest split-K factor of a projection.
constexpr int GEMM_MAX_SPLITS = 32;

// Epilogue of a projection (see k_gemm.hip).
enum { GEMM_EPI_STORE = 0,      // C[r][n] = y
       GEMM_EPI_RESIDUAL = 1,   // x[r][n] += y
       GEMM_EPI_SWIGLU = 2,     // columns packed [16 gate | 16 up] per 32; act[r][f] = silu(g) * u
       GEMM_EPI_QKV = 3,        // RoPE; q -> q_out, k and v -> the row's KV page
       GEMM_EPI_PARTIAL = 4 };  // (internal) split partial to part[s]
struct GemmEpi {
  int mode;
  float* C; int ldc;                      // STORE
  float* x; int ldx;                      // RESIDUAL
  const float* norm_g; float norm_eps; ActOut norm_out;   // RESIDUAL with K split: then RMSNorm the row
                                                          // into norm_out (ignored without a split)
  ActOut act; int act_ld;                 // SWIGLU
  float* q_out; void* kv_pool; KvGeom geom; int layer;      // QKV
  const int32_t* page_tab; int tab_stride; const int32_t* row_tab; const int32_t* row_pos;
  const float* rope_cos; const float* rope_sin; int n_q, n_kv, hd;
  float* part; int64_t part_stride;       // split partials [S][rows][N] (S > 1 and fp32 models)
};

// y = A W^T over rows < *d_rows with K split `splits` ways (bf16 models: K
// and k_per_split multiples of 64, N a multiple of 16; fp32 models: one
// split), then the epilogue ep.
hipError_t launch_gemm(int dtype, const void* A, int lda, int64_t a_plane, const void* W, int ldw, const int* d_rows,
                       int rows_ub, int N, int K, int splits, int k_per_split, const GemmEpi& ep, hipStream_t st);

// x[r] = embed[tok[r]] (fp32), r < *d_rows.  Prefill: tok = prompts.  An id
// outside [0, V) reads row 0 instead and sets *bad_token = 1.
hipError_t launch_embed(int dtype, const void* embed, int d, int V, const int32_t* tok, float* x,
                        int32_t* bad_token, const int* d_rows, int rows_ub, hipStream_t st);

// Decode row setup for step t = *d_t >= 1: row r (< *d_rows) feeds act_tok[r]
// for sequence s = act_seq[r] at position plen[grp[s]] + t - 1; writes
// row_tab, row_pos, row_beg (the prompt's full-page length when
// prefix_split, else 0) and the embedded token into x.
hipError_t launch_decode_rows(int dtype, const void* embed, int d, const int32_t* act_seq,
                              const int32_t* act_tok, const int32_t* seq_grp, const int32_t* plen, const int* d_t,
                              int prefix_split, int32_t* row_tab, int32_t* row_pos, int32_t* row_beg, float* x,
                              const int* d_rows, int rows_ub, hipStream_t st);

// Prefill row setup: row r belongs to prompt p with prompt_off[p] <= r <
// prompt_off[p+1]; row_tab[r] = tab_base + p, row_pos[r] = r - prompt_off[p],
// row_beg[r] = 0.
hipError_t launch_prefill_rows(const int32_t* prompt_off, int P, int tab_base, int32_t* row_tab,
                               int32_t* row_pos, int32_t* row_beg, int total, hipStream_t st);

// out[r] = x[r] / sqrt(mean(x[r]^2) + eps) * g as an activation operand.  If
// src_rows != NULL the input row is x[src_rows[r]].
hipError_t launch_rmsnorm(int dtype, const float* x, const float* g, int d, float eps, void* out, int64_t a_plane,
                          const int32_t* src_rows, const int* d_rows, int rows_ub, hipStream_t st);

// Partial slots of the attention of one row: slots 0..pre_slots-1 take the
// shared-prefix chunks of pre_chunk tokens (prefix pass), slots
// pre_slots..n_slots-1 the row's own n_chunks chunks (per-row pass).
struct AttPlan {
  int n_chunks;    // per-row chunks
  int pre_slots;   // prefix chunks (0: no prefix pass)
  int pre_chunk;   // tokens per prefix chunk, a multiple of 32
  int n_slots;     // pre_slots + n_chunks
};

// bf16 models whose rows take 2..8 context chunks (and no prefix pass) run one
// workgroup per (row, kv head) whose waves merge the chunks themselves:
// launch_attention then writes the activation and no merge launch follows.
// Only where rows_ub * n_kv gives every CU a workgroup: with fewer, the
// per-chunk grid plus a merge launch keeps more CUs busy and is faster.
inline bool att_merges_in_kernel(int dtype, const AttPlan& plan, int rows_ub, int n_kv) {
  return dtype == 1 && plan.pre_slots == 0 && plan.n_chunks >= 2 && plan.n_chunks <= 8 &&
         (int64_t)rows_ub * n_kv >= 256;
}

// Per-row pass.  Row r covers positions row_beg[r]..row_pos[r] of page table
// row_tab[r] (at most max_ctx tokens), cut into n_chunks equal chunks
// (rounded up to 32 tokens); each (row, kv head, chunk) work item writes a
// partial (max, sum, unnormalised output) per query head.  row_beg[r] is a
// multiple of 16.  bf16 models with a single slot (plan.n_slots == 1) write
// the normalised output straight into the activation planes `out` instead
// (no merge needed).
hipError_t launch_attention(int dtype, const float* q, int n_q, int n_kv, int head_dim,
                            const void* kv_pool, KvGeom g, int layer, const int32_t* page_tab,
                            int tab_stride, const int32_t* row_tab, const int32_t* row_pos, const int32_t* row_beg,
                            int max_ctx, AttPlan plan, float* part_o, float* part_ml, void* out, int64_t a_plane,
                            const int* d_rows, int rows_ub, hipStream_t st);

// Prefix pass (bf16 models).  The active rows of prompt p are grp_row0[p] ..
// grp_row1[p]-1 (empty when equal); all of them attend to positions
// 0..(plen[p]/16)*16-1 of page table row tab_base + p, which every row of the
// group has as its row_beg.  max_group_rows bounds grp_row1[p] - grp_row0[p].
hipError_t launch_attention_prefix(const float* q, int n_q, int n_kv, int head_dim, const void* kv_pool, KvGeom g,
                                   int layer, const int32_t* page_tab, int tab_stride, int tab_base,
                                   const int32_t* plen, const int32_t* grp_row0, const int32_t* grp_row1, int P,
                                   int max_group_rows, AttPlan plan, float* part_o, float* part_ml, hipStream_t st);

// Row-tile pass (bf16 models, prefill-style rows): tile k = rows tile_r0[k] ..
// + tile_nr[k] - 1 (at most att_tile_rows) of one page table row at consecutive
// positions; every query row attends causally to positions 0..row_pos of its
// row and the normalised output goes to the activation planes `out`.
// *d_tiles <= tiles_ub tiles; max_ctx bounds every row's context.
hipError_t launch_attention_tile(const float* q, int n_q, int n_kv, int head_dim, const void* kv_pool, KvGeom g,
                                 int layer, const int32_t* page_tab, int tab_stride, const int32_t* row_tab,
                                 const int32_t* row_pos, const int32_t* tile_r0, const int32_t* tile_nr,
                                 const int* d_tiles, int tiles_ub, int max_ctx, void* out, int64_t a_plane,
                                 hipStream_t st);

// Merge the partial slots of each (row, q head) into the activation operand
// out [rows][n_q*head_dim].
hipError_t launch_attn_merge(int dtype, const float* part_o, const float* part_ml, int n_q,
                             int head_dim, const int32_t* row_pos, const int32_t* row_beg, AttPlan plan, void* out,
                             int64_t a_plane, const int* d_rows, int rows_ub, hipStream_t st);

struct SampleArgs {
  const float* logits;      // [rows][V] or [P][V] when logits_by_group
  int logits_by_group;      // step 0: logits row = seq_grp[s]
  int V, eos, max_new;
  const int* d_t;           // device step index
  uint64_t seed;
  float temperature;
  const int32_t* act_seq;   // row -> sequence
  const int32_t* seq_grp;
  const int32_t* forced_len;   // device [N] or NULL
  const int32_t* force_tokens; // device [N*max_new] or NULL
  float* dump_logits; int dump_steps; int n_seq;
  int32_t* tokens_out; float* logprobs_out;
  int32_t* next_tok;        // [rows] token fed to the next step
  int32_t* done;            // [rows]
  int32_t* bad_token;       // set to 1 when a forced token id is outside [0, V)
  const int* d_rows;
  float* part;              // [rows][n_slices][4] slice partials
  int n_slices;             // vocabulary slices per row
};
hipError_t launch_sample(const SampleArgs& a, int rows_ub, hipStream_t st);

// Retire/compact after the step whose index is state[8]; advances state[8].
// Also publishes each prompt's range of rows among the surviving ones
// (grp_row0[p] .. grp_row1[p]-1; compaction keeps rows in sequence order).
struct CompactArgs {
  int max_new, page_tok, max_pages, n_seq, P;
  int32_t* grp_row0; int32_t* grp_row1;
  int32_t* act_seq; int32_t* act_tok; const int32_t* done;
  const int32_t* seq_grp; const int32_t* plen;
  int32_t* page_tab; int32_t* seq_npages; const int32_t* seq_nshared;
  int32_t* free_stack;
  int32_t* state;     // [0] active rows, [1] free-stack top, [2] out-of-pages flag, [8] step
  int32_t* lengths;
  int32_t* hist_active; int32_t* hist_groups; int64_t* hist_ctx; int hist_cap;
};
hipError_t launch_compact(const CompactArgs& a, hipStream_t st);

struct ForkArgs {
  int P, n_seq, page_tok, max_pages, share;
  const int32_t* grp_off;   // [P+1]
  const int32_t* plen;      // [P]
  int32_t* page_tab;        // rows 0..n_seq-1 sequences, n_seq+p prompt tables
  int32_t* seq_grp; int32_t* seq_npages; int32_t* seq_nshared;
  int32_t* act_seq;
  int32_t* free_stack; int32_t* state;
  int32_t* copy_pairs;      // out: [2*k] (src page, dst page); count in state[3]
};
hipError_t launch_fork(const ForkArgs& a, hipStream_t st);
hipError_t launch_page_copy(int dtype, void* kv_pool, const KvGeom& g, const int32_t* copy_pairs,
                            int max_pairs, const int32_t* state, hipStream_t st);

// Rollout set-up: prompt tables, free stack, output padding, counters.
struct SetupArgs {
  int P, n_seq, max_new, page_tok, max_pages;
  int64_t pool_pages;
  const int32_t* plen; int32_t* prompt_off; int32_t* grp_off; const int32_t* G;
  int32_t* page_tab; int32_t* free_stack; int32_t* state;
  int32_t* tokens_out; float* logprobs_out;
  int32_t* last_rows;      // [P] row of each prompt's last token
  // state: [0] active rows, [1] free-stack top, [2] out-of-pages flag, [3] page
  // copies pending, [4] prefix pages, [5] prompt tokens, [6] prompts, [7] invalid token id seen,
  // [8] step index
};
hipError_t launch_setup(const SetupArgs& a, hipStream_t st);

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t st);

// Per-group length summaries for the group-size controller: stats[p] =
// (l_max, l_median, l_max / l_median, [l_max / l_median > tau]) of group p's
// lengths (prompt-major, group sizes G, 1 <= G[p] <= 1024); NaN for a group
// outside the bounds.
hipError_t launch_group_stats(const int32_t* lengths, const int32_t* G, int P, int N, double tau, float* stats,
                              hipStream_t st);

hipError_t launch_group_filter(const float* rewards, const int32_t* G, int P, int N, int32_t* keep, int32_t* kept_ids,
                               int32_t* n_kept, hipStream_t st);
hipError_t launch_group_advantage(const float* rewards, const int32_t* G, int P, int N, float eps,
                                  int ddof, float* adv, hipStream_t st);
hipError_t launch_philox_blocks(uint64_t k0, uint64_t k1, const uint64_t* ctr, int64_t n, uint64_t* out,
                                hipStream_t st);
hipError_t launch_gumbel_bits(uint64_t seed, int t, int s, int vocab, uint32_t* out, hipStream_t st);
// Streaming ceiling probe: mode 1 copies `bytes` from src to dst, mode 0 only
// reads src and stores one word per thread (blocks*256 words) to dst.
hipError_t launch_hbm_probe(const void* src, void* dst, int64_t bytes, int mode, int blocks, hipStream_t st);

// ---- GRPO loss forward (k_loss.hip)
// After the fork: per-sequence row offsets of the teacher-forced forward
// (coff [n_seq + 1], prefix of lengths - 1) and the pages its positions need.
// state[9] = rows in all, state[10] = length out of [1, max_new] seen,
// state[2] = out of pages.
struct ReserveArgs {
  int n_seq, max_new, page_tok, max_pages;
  const int32_t* lengths; const int32_t* plen; const int32_t* seq_grp;
  int32_t* seq_npages; int32_t* page_tab; const int32_t* free_stack;
  int32_t* coff; int32_t* state;
};
hipError_t launch_reserve(const ReserveArgs& a, hipStream_t st);

// Rows row0 .. row0 + rows - 1 of the teacher-forced forward: row set-up
// (row_tab, row_pos, row_beg), embeddings into x, and for each row the token
// it predicts (row_tgt) and where that token's log-probability goes (row_out).
struct RecomputeRows {
  int row0, n_seq, max_new, V, d;
  const int32_t* coff; const int32_t* tokens; const int32_t* plen; const int32_t* seq_grp;
  int32_t* row_tab; int32_t* row_pos; int32_t* row_beg; int32_t* row_tgt; int32_t* row_out;
  float* x; int32_t* bad_token;
};
hipError_t launch_recompute_rows(int dtype, const void* embed, const RecomputeRows& a, int rows, hipStream_t st);
// Cuts rows 0..n-1 of a recompute chunk (row_tab = sequence, coff = row
// offsets, row0 = the chunk's first global row) into per-sequence tiles of at
// most 16 rows for the row-tile attention.
hipError_t launch_row_tiles(const int32_t* row_tab, const int32_t* coff, int row0, int n, int tile_rows,
                            int32_t* tile_r0, int32_t* tile_nr, int* d_tiles, hipStream_t st);
// Positions per row tile the row-tile attention takes for this GQA shape.
int att_tile_rows(int n_q, int n_kv);
// Work items (waves) a per-row attention launch aims for.
constexpr int ATT_ITEMS_TARGET = 1024;
// Context chunks per row for a per-row attention launch over rows_ub rows
// whose contexts are at most ctx_max tokens.
int att_row_chunks(int rows_ub, int n_kv, int ctx_max);
hipError_t launch_first_rows(const int32_t* tokens, const int32_t* seq_grp, int n_seq, int max_new, int V,
                             int32_t* lrow, int32_t* tgt, int32_t* out, int32_t* bad_token, hipStream_t st);
// lp[out[r]] = z[tgt[r]]/T - logsumexp(z/T), z = logits row lrow[r] (lrow NULL: r).
hipError_t launch_token_logprob(const float* logits, int V, float T, const int32_t* lrow, const int32_t* tgt,
                                const int32_t* out, float* lp, int rows, hipStream_t st);

struct SurrogateArgs {
  const float* new_lp; const float* old_lp; const float* adv; const int32_t* lengths;
  const int32_t* G; const int32_t* keep;
  int P, N, max_new, mode;
  double eps_lo, eps_hi;
  double* out;
};
// Per-sequence record of the clipped surrogate's first pass (16 bytes):
// the fp64 sum of the sequence's terms and its clipped-token count (-1 for a
// length outside [1, max_new]).
struct SurrogateRec {
  double acc;
  int32_t clips;
  int32_t pad;
};
static_assert(sizeof(SurrogateRec) == 16, "surrogate record layout");
// Two launches: per-sequence records into rec [N] (device scratch), then one
// block that reduces them in a fixed order into a.out.
hipError_t launch_surrogate(const SurrogateArgs& a, SurrogateRec* rec, hipStream_t st);
// Largest N of grpo_surrogate_noalloc: its records live in a static device
// array of this many entries (k_loss.hip).
constexpr int SURROGATE_NOALLOC_MAX_SEQS = 65536;
// Device address of that array on the current device (looked up with
// hipGetSymbolAddress on the first call per device, then cached).
hipError_t surrogate_static_scratch(SurrogateRec** out);
