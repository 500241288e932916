// Host side of librollout.so: policy creation (weight repacking, workspace
// arena, KV page pool), the rollout driver and the C ABI declared in
// include/rollout.h.
//
// Rollout driver.  Prefill runs every prompt once over all prompt tokens as
// one batch of rows, writing keys/values into the prompt's KV pages; the lm
// head runs on each prompt's last position.  The fork gives every sibling the
// prompt's full pages by reference.  Step 0 samples every sibling from its
// prompt's logits; step t >= 1 feeds each active sequence's previous token
// through the decoder.  After each step one kernel retires finished rows and
// compacts the survivors; the active count is copied back asynchronously and
// the host sizes later grids with the last count it has seen (an upper bound,
// since the count never grows), running at most RG_LOOKAHEAD steps ahead.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

#include "rollout.h"
#include "rg_kernels.h"

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIPTRY(expr)                                                                         \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(RG_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr int RG_PAGE_TOK = 16;        // tokens per KV page
constexpr int RG_SPLIT_MAX = GEMM_MAX_SPLITS;   // largest split-K factor of a decode GEMM
constexpr int RG_GEMM_TARGET = 384;    // blocks a split-K GEMM launch aims for
constexpr int RG_GEMM_FULL = 256;      // output-tile blocks that need no split
constexpr int RG_PRE_TARGET = 512;     // workgroups the prefix attention pass aims for
constexpr int RG_PRE_MIN_CHUNK = 64;   // fewest prefix tokens per prefix workgroup
constexpr int RG_PRE_MAX_SLOTS = 16;   // prefix chunks per row (more only for prefixes > 16k tokens)
constexpr int RG_RING = 64;            // async active-count slots
constexpr int RG_LOOKAHEAD = 4;        // decode steps enqueued beyond the last seen count
constexpr int RG_PROF_RING = 8192;     // event pairs in flight when profiling
constexpr int RG_SAMPLE_SLICES_MAX = 32;  // vocabulary slices per sampled row
constexpr int RG_LM_SLICE_ROWS = 2048;    // recompute: lm-head rows per slice (when the activations hold them)
constexpr int RG_PROF_PHASES = 2 + 8;     // prefill, decode, decode by row bucket (16 .. 512, larger)

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

struct rg_policy {
  rg_config cfg{};
  rg_limits lim{};
  int dtype = 0;
  size_t eb = 4;
  int d = 0, V = 0, L = 0, F = 0, hd = 0, nq = 0, nkv = 0, q_dim = 0, kv_dim = 0, qkv_n = 0;
  int page_tok = RG_PAGE_TOK, max_pages = 0, m_act = 0;
  KvGeom geom{};

  void* w_embed = nullptr;
  float* w_final = nullptr;
  void* w_lm = nullptr;
  std::vector<void*> w_qkv, w_o, w_gu, w_down;
  std::vector<float*> g_attn, g_ffn;
  float* rope_cos = nullptr;
  float* rope_sin = nullptr;

  void* kv_pool = nullptr;
  int64_t pool_pages = 0;

  float* x = nullptr;
  void* abuf = nullptr;   // activation operand (ping)
  void* abuf2 = nullptr;  // activation operand (pong)
  int64_t a_plane = 0;   // elements between the hi and lo planes of abuf (bf16 models)
  float* cpart = nullptr;
  int64_t cpart_elems = 0;
  float* qbuf = nullptr;
  float* att_o = nullptr;
  float* att_ml = nullptr;
  int64_t att_rowchunks = 0;
  int64_t logit_rows = 0;   // rows of the fp32 logits buffer
  float* logits = nullptr;
  float* sample_part = nullptr;   // [rows][RG_SAMPLE_SLICES_MAX][4]
  int32_t *page_tab = nullptr, *seq_grp = nullptr, *seq_npages = nullptr, *seq_nshared = nullptr,
          *seq_forced = nullptr, *grp_off = nullptr, *prompt_off = nullptr, *plen = nullptr, *G_dev = nullptr,
          *act_seq = nullptr, *act_tok = nullptr, *done = nullptr, *row_tab = nullptr, *row_pos = nullptr,
          *free_stack = nullptr, *state = nullptr, *copy_pairs = nullptr, *last_rows = nullptr,
          *hist_active = nullptr, *hist_groups = nullptr, *row_beg = nullptr, *grp_row0 = nullptr,
          *grp_row1 = nullptr, *coff = nullptr, *row_tgt = nullptr, *row_out = nullptr, *row_lrow = nullptr,
          *tile_r0 = nullptr, *tile_nr = nullptr;
  int64_t* hist_ctx = nullptr;
  int hist_cap = 0;

  int32_t* h_stage = nullptr;  // pinned staging for host inputs
  int32_t* h_ring = nullptr;   // pinned [RG_RING][8] state snapshots
  hipEvent_t ring_ev[RG_RING]{};

  std::vector<void*> allocs;
  int64_t dev_bytes = 0;

  // profiling
  bool prof = false;
  uint32_t prof_mask = 0xFFFFFFFFu;
  int prof_phase = 0;
  std::vector<hipEvent_t> prof_ev;  // 2 * RG_PROF_RING
  std::vector<int> prof_kind, prof_ph;
  int64_t prof_head = 0, prof_tail = 0;
  // [0] prefill, [1] decode (all steps), [2 + b] decode steps of row bucket b
  double kt_ms[RG_PROF_PHASES][RG_K_COUNT]{};
  int64_t kt_n[RG_PROF_PHASES][RG_K_COUNT]{};

  int32_t last_steps = 0;
  hipEvent_t phase_ev[3]{};   // start of prefill, end of prefill + fork, end of decode (last rollout_group)
  bool phase_valid = false;

  hipStream_t cap_st = nullptr;   // private stream used only to capture decode-step graphs
  bool use_graphs = true;
  int progress_every = 0;   // RG_PROGRESS=N: a stderr line every N enqueued decode steps

  int alloc(void** p, size_t bytes) {
    bytes = std::max<size_t>(bytes, 256);
    hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) return fail(e == hipErrorOutOfMemory ? RG_ENOMEM : RG_EHIP,
                                     "hipMalloc(" + std::to_string(bytes) + "): " + hipGetErrorString(e));
    allocs.push_back(*p);
    dev_bytes += (int64_t)bytes;
    return RG_OK;
  }
  ~rg_policy() {
    for (void* p : allocs) (void)hipFree(p);
    if (h_stage) (void)hipHostFree(h_stage);
    if (h_ring) (void)hipHostFree(h_ring);
    for (auto& e : ring_ev) if (e) (void)hipEventDestroy(e);
    for (auto& e : prof_ev) if (e) (void)hipEventDestroy(e);
    for (auto& e : phase_ev) if (e) (void)hipEventDestroy(e);
    if (cap_st) (void)hipStreamDestroy(cap_st);
  }
};

// Error reporting for the other host sources of the library.
int rg_set_error(int code, const char* msg) { return fail(code, msg); }

// ---------------------------------------------------------------- launch-event hook
namespace {
thread_local hipEvent_t g_arm_start = nullptr, g_arm_stop = nullptr;
}
void rg_arm_launch_events(hipEvent_t start, hipEvent_t stop) { g_arm_start = start; g_arm_stop = stop; }
bool rg_take_launch_events(hipEvent_t* start, hipEvent_t* stop) {
  if (!g_arm_start) return false;
  *start = g_arm_start;
  *stop = g_arm_stop;
  g_arm_start = g_arm_stop = nullptr;
  return true;
}
bool rg_launch_events_armed() { return g_arm_start != nullptr; }

namespace {

// ---------------------------------------------------------------- profiling
int prof_drain_one(rg_policy* p) {
  const int64_t i = p->prof_tail % RG_PROF_RING;
  HIPTRY(hipEventSynchronize(p->prof_ev[2 * i + 1]));
  float ms = 0.f;
  HIPTRY(hipEventElapsedTime(&ms, p->prof_ev[2 * i], p->prof_ev[2 * i + 1]));
  const int ph = p->prof_ph[i], k = p->prof_kind[i];
  p->kt_ms[ph][k] += ms;
  p->kt_n[ph][k] += 1;
  if (ph >= 2) {   // a decode step of one row bucket also counts towards the decode total
    p->kt_ms[1][k] += ms;
    p->kt_n[1][k] += 1;
  }
  p->prof_tail++;
  return RG_OK;
}

// Times one launcher call of a kernel class.  Bracketing: events recorded on
// the stream before and after the call (every class; includes the stream's
// dispatch overhead).  Dispatch (ext = true, single-kernel launchers that
// take armed events): the events are the kernel dispatch's own timestamps.
struct ProfScope {
  rg_policy* p;
  hipStream_t st;
  int64_t slot = -1;
  bool ext = false;
  int rc = RG_OK;
  ProfScope(rg_policy* pol, hipStream_t s, int kind, bool dispatch_events) : p(pol), st(s) {
    if (!p->prof || !((p->prof_mask >> kind) & 1u)) return;
    if (p->prof_head - p->prof_tail >= RG_PROF_RING) rc = prof_drain_one(p);
    slot = p->prof_head % RG_PROF_RING;
    p->prof_kind[slot] = kind;
    p->prof_ph[slot] = p->prof_phase;
    ext = dispatch_events;
    if (ext) rg_arm_launch_events(p->prof_ev[2 * slot], p->prof_ev[2 * slot + 1]);
    else (void)hipEventRecord(p->prof_ev[2 * slot], st);
  }
  ~ProfScope() {
    if (slot < 0) return;
    if (ext) {
      if (rg_launch_events_armed()) {   // the launcher launched nothing
        hipEvent_t a, b;
        rg_take_launch_events(&a, &b);
        return;
      }
    } else {
      (void)hipEventRecord(p->prof_ev[2 * slot + 1], st);
    }
    p->prof_head++;
  }
};

#define LAUNCH_(kind, call, ext)                                                              \
  do {                                                                                        \
    ProfScope ps_(pol, st, kind, ext);                                                        \
    if (ps_.rc != RG_OK) return ps_.rc;                                                        \
    hipError_t e_ = (call);                                                                   \
    if (e_ != hipSuccess) return fail(RG_EHIP, std::string("launch ") + #kind + ": " + hipGetErrorString(e_)); \
  } while (0)
#define LAUNCH(kind, call) LAUNCH_(kind, call, false)
// single-kernel launchers that time their dispatch with armed events
#define LAUNCH_TIMED(kind, call) LAUNCH_(kind, call, true)

// Split-K factor of a projection: enough blocks to cover the chip, each
// split at least two 64-wide K steps, and the fp32 split partials (written
// once, read once by the reducing block) within max(2 x weight bytes, 32 MB).
void choose_splits(const rg_policy* pol, int N, int rows_ub, int K, int* splits, int* kps) {
  int S = 1;
  if (pol->dtype == RG_DTYPE_BF16) {
    // Split K only while the output tiles leave the chip short of blocks, to
    // about RG_GEMM_TARGET blocks (twice that for narrow outputs, whose
    // partials are small), and only as far as the fp32 partials (written
    // once, read once: 8 bytes per output element and split) stay within
    // twice the weight bytes or 24 MiB.
    const int64_t bm = gemm_tile_rows(pol->dtype, rows_ub, N), bn = gemm_tile_cols(pol->dtype, rows_ub, N, K);
    const int64_t blocks = ceil_div(N, bn) * ceil_div(rows_ub, bm);
    const int64_t target = N >= 8192 ? RG_GEMM_TARGET : 2 * RG_GEMM_TARGET;
    if (blocks < RG_GEMM_FULL) S = (int)ceil_div(target, blocks);
    const int64_t budget = std::max<int64_t>(4LL * N * K, 24LL << 20);
    S = (int)std::min<int64_t>({(int64_t)S, K / 128, budget / (8LL * rows_ub * N), RG_SPLIT_MAX});
    S = std::max(1, S);
  }
  const int step = pol->dtype == RG_DTYPE_BF16 ? 64 : 1;
  int k = (int)(ceil_div(ceil_div(K, S), step) * step);
  *kps = k;
  *splits = (int)ceil_div(K, k);
}

// Split plan of a projection into the split-K workspace.
void plan(const rg_policy* pol, int N, int rows_ub, int K, int* S, int* kps) {
  choose_splits(pol, N, rows_ub, K, S, kps);
  const int64_t fit = pol->cpart_elems / ((int64_t)rows_ub * N);   // splits the workspace holds
  if (*S > fit) {
    const int step = pol->dtype == RG_DTYPE_BF16 ? 64 : 1;
    *S = (int)std::max<int64_t>(1, fit);
    *kps = (int)ceil_div(ceil_div(K, *S), step) * step;
    *S = (int)ceil_div(K, *kps);
  }
}

// One projection with its epilogue; the split plan and workspace are filled in here.
int gemm(rg_policy* pol, hipStream_t st, int kind, const void* A, int K, const void* W, int N, const int* d_rows,
         int rows_ub, GemmEpi ep, bool allow_split = true, int* splits_out = nullptr) {
  int S = 1, kps = K;
  if (allow_split) plan(pol, N, rows_ub, K, &S, &kps);
  if (splits_out) *splits_out = S;
  ep.part = pol->cpart;
  ep.part_stride = (int64_t)rows_ub * N;
  const bool needs_part = S > 1 || pol->dtype != RG_DTYPE_BF16;
  if (needs_part && ep.part_stride * S > pol->cpart_elems) return fail(RG_ENOMEM, "GEMM workspace too small");
  LAUNCH(kind, launch_gemm(pol->dtype, A, K, pol->a_plane, W, K, d_rows, rows_ub, N, K, S, kps, ep, st));
  return RG_OK;
}

// With RG_FLAG_GROUP_PREFIX, decode steps of bf16 models attend to each
// prompt's full prefix pages once per group (prefix pass) and to the rest per
// row.
struct PrefixPass {
  int P;                // prompts
  int tab_base;         // page table row of prompt 0 (the rollout's N)
  int max_group_rows;   // largest G
  int max_pref;         // largest full-page prefix, (plen / 16) * 16
};

// Row tiles of prefill-style rows (bf16 models): attention by the row-tile
// pass instead of the per-row pass.
struct RowTiles {
  const int* d_tiles;   // tile count on the device
  int tiles_ub;         // bound on it, sizes the grid
};

// The decoder blocks over `rows_ub` rows (actual count at *d_rows), whose
// row_tab / row_pos / row_beg are set and whose first attention norm is in
// pol->abuf; ctx_max bounds every row's context length.  pre != NULL runs the
// prefix pass (row_beg then holds each row's prefix length).  On return
// pol->abuf holds the final norm of every row (final_norm_rows) or x the
// residual stream after the last block.
int run_layers(rg_policy* pol, hipStream_t st, const int* d_rows, int rows_ub, int ctx_max, bool final_norm_rows,
               const PrefixPass* pre, const RowTiles* tiles = nullptr) {
  if (rows_ub <= 0) return RG_OK;
  const int tab_stride = pol->max_pages;
  const int n_chunks = att_row_chunks(rows_ub, pol->nkv, ctx_max);
  AttPlan plan{n_chunks, 0, 0, n_chunks};
  if (pre && pre->max_pref > 0) {
    // prefix chunks: about RG_PRE_TARGET workgroups, at least RG_PRE_MIN_CHUNK
    // tokens and at most 1024 tokens each
    int slots = (int)std::min<int64_t>({ceil_div(RG_PRE_TARGET, (int64_t)pol->nkv * pre->P),
                                        ceil_div(pre->max_pref, RG_PRE_MIN_CHUNK), RG_PRE_MAX_SLOTS});
    slots = std::max<int>({1, slots, (int)ceil_div(pre->max_pref, 1024)});
    plan.pre_chunk = (int)ceil_div(ceil_div(pre->max_pref, slots), 32) * 32;
    plan.pre_slots = (int)ceil_div(pre->max_pref, plan.pre_chunk);
    plan.n_slots = plan.pre_slots + n_chunks;
  }
  if (!tiles && (int64_t)rows_ub * plan.n_slots > pol->att_rowchunks)
    return fail(RG_ENOMEM, "attention workspace too small");
  const float eps = pol->cfg.rms_eps;
  GemmEpi qkv{};
  qkv.mode = GEMM_EPI_QKV;
  qkv.q_out = pol->qbuf; qkv.kv_pool = pol->kv_pool; qkv.geom = pol->geom;
  qkv.page_tab = pol->page_tab; qkv.tab_stride = tab_stride; qkv.row_tab = pol->row_tab; qkv.row_pos = pol->row_pos;
  qkv.rope_cos = pol->rope_cos; qkv.rope_sin = pol->rope_sin; qkv.n_q = pol->nq; qkv.n_kv = pol->nkv; qkv.hd = pol->hd;
  GemmEpi resid{};
  resid.mode = GEMM_EPI_RESIDUAL; resid.x = pol->x; resid.ldx = pol->d;
  resid.norm_eps = eps; resid.norm_out = ActOut{pol->abuf, pol->a_plane};
  GemmEpi swig{};
  swig.mode = GEMM_EPI_SWIGLU; swig.act = ActOut{pol->abuf2, pol->a_plane}; swig.act_ld = pol->F;
  int rc;

  for (int l = 0; l < pol->L; ++l) {
    qkv.layer = l;
    if ((rc = gemm(pol, st, RG_K_GEMM_QKV, pol->abuf, pol->d, pol->w_qkv[l], pol->qkv_n, d_rows, rows_ub, qkv)))
      return rc;
    if (tiles) {
      LAUNCH_TIMED(RG_K_ATTN, launch_attention_tile(pol->qbuf, pol->nq, pol->nkv, pol->hd, pol->kv_pool, pol->geom, l,
                                                    pol->page_tab, tab_stride, pol->row_tab, pol->row_pos,
                                                    pol->tile_r0, pol->tile_nr, tiles->d_tiles, tiles->tiles_ub,
                                                    ctx_max, pol->abuf2, pol->a_plane, st));
    } else {
    if (plan.pre_slots)
      LAUNCH_TIMED(RG_K_ATTN, launch_attention_prefix(pol->qbuf, pol->nq, pol->nkv, pol->hd, pol->kv_pool, pol->geom, l,
                                                pol->page_tab, tab_stride, pre->tab_base, pol->plen,
                                                pol->grp_row0, pol->grp_row1, pre->P, pre->max_group_rows, plan,
                                                pol->att_o, pol->att_ml, st));
    LAUNCH_TIMED(RG_K_ATTN, launch_attention(pol->dtype, pol->qbuf, pol->nq, pol->nkv, pol->hd, pol->kv_pool, pol->geom, l,
                                       pol->page_tab, tab_stride, pol->row_tab, pol->row_pos, pol->row_beg, ctx_max,
                                       plan, pol->att_o, pol->att_ml, pol->abuf2, pol->a_plane, d_rows, rows_ub, st));
    // one bf16 slot, or chunks merged inside the attention kernel: it wrote abuf2 itself
    if ((plan.n_slots > 1 && !att_merges_in_kernel(pol->dtype, plan, rows_ub, pol->nkv)) || pol->dtype != RG_DTYPE_BF16)
      LAUNCH(RG_K_ATTN_MERGE, launch_attn_merge(pol->dtype, pol->att_o, pol->att_ml, pol->nq, pol->hd, pol->row_pos,
                                                pol->row_beg, plan, pol->abuf2, pol->a_plane, d_rows, rows_ub, st));
    }
    // O projection + residual, then the MLP norm into abuf (fused into the
    // split epilogue when K is split)
    int S;
    resid.norm_g = pol->g_ffn[l];
    if ((rc = gemm(pol, st, RG_K_GEMM_O, pol->abuf2, pol->q_dim, pol->w_o[l], pol->d, d_rows, rows_ub, resid, true, &S)))
      return rc;
    if (S == 1 || pol->dtype != RG_DTYPE_BF16)
      LAUNCH(RG_K_RMSNORM, launch_rmsnorm(pol->dtype, pol->x, pol->g_ffn[l], pol->d, eps, pol->abuf, pol->a_plane,
                                           nullptr, d_rows, rows_ub, st));
    if ((rc = gemm(pol, st, RG_K_GEMM_GU, pol->abuf, pol->d, pol->w_gu[l], 2 * pol->F, d_rows, rows_ub, swig)))
      return rc;
    const float* gnext = l + 1 < pol->L ? pol->g_attn[l + 1] : (final_norm_rows ? pol->w_final : nullptr);
    resid.norm_g = gnext;
    if ((rc = gemm(pol, st, RG_K_GEMM_DOWN, pol->abuf2, pol->F, pol->w_down[l], pol->d, d_rows, rows_ub, resid, true,
                   &S)))
      return rc;
    if (gnext && (S == 1 || pol->dtype != RG_DTYPE_BF16))
      LAUNCH(RG_K_RMSNORM, launch_rmsnorm(pol->dtype, pol->x, gnext, pol->d, eps, pol->abuf, pol->a_plane, nullptr,
                                           d_rows, rows_ub, st));
  }
  return RG_OK;
}

// The lm head into pol->logits.  src_rows != NULL (prefill): final norm of the
// listed rows first; otherwise pol->abuf already holds the final norm.
int run_head(rg_policy* pol, hipStream_t st, const int* d_rows, int rows_ub, const int32_t* src_rows) {
  if (src_rows)
    LAUNCH(RG_K_RMSNORM, launch_rmsnorm(pol->dtype, pol->x, pol->w_final, pol->d, pol->cfg.rms_eps, pol->abuf,
                                         pol->a_plane, src_rows, d_rows, rows_ub, st));
  GemmEpi store{};
  store.mode = GEMM_EPI_STORE; store.C = pol->logits; store.ldc = pol->V;
  return gemm(pol, st, RG_K_GEMM_LM, pol->abuf, pol->d, pol->w_lm, pol->V, d_rows, rows_ub, store, false);
}

// Row bound used for a decode step: the host's bound rounded up, so that the
// few distinct bounds share split plans and captured graphs.
int row_bucket(int m) {
  if (m <= 16) return 16;
  if (m <= 32) return 32;
  if (m <= 64) return 64;
  if (m <= 128) return 128;
  if (m <= 256) return 256;
  if (m <= 384) return 384;
  return (int)ceil_div(m, 256) * 256;
}

// Profiling phase of a decode step with row bound rows_ub: 2 + the index of
// its row bucket (16, 32, 64, 128, 256, 384, 512, larger).
int bucket_phase(int rows_ub) {
  const int edges[7] = {16, 32, 64, 128, 256, 384, 512};
  int b = 0;
  while (b < 7 && rows_ub > edges[b]) ++b;
  return 2 + b;
}

// Vocabulary slices per sampled row: about 4096 blocks in all, at most
// RG_SAMPLE_SLICES_MAX per row (the slice scan is bound by its vector ALU
// work; more, shorter slices hide its latency better: 1.5B sampler per group
// step 309 ms at 1024 blocks, 281 at 2048, 271 at 4096).
int sample_slices(int rows_ub) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(RG_SAMPLE_SLICES_MAX, ceil_div(4096, std::max(1, rows_ub))));
}

// Every kernel of one decode step (t >= 1, read on the device from state[8]).
int enqueue_step(rg_policy* pol, hipStream_t st, int rows_ub, int ctx_max, SampleArgs sm, const CompactArgs& ca,
                 const PrefixPass* pre) {
  sm.n_slices = sample_slices(rows_ub);
  int rc;
  LAUNCH(RG_K_EMBED, launch_decode_rows(pol->dtype, pol->w_embed, pol->d, pol->act_seq, pol->act_tok, pol->seq_grp,
                                        pol->plen, pol->state + 8, pre ? 1 : 0, pol->row_tab, pol->row_pos,
                                        pol->row_beg, pol->x, pol->state, rows_ub, st));
  LAUNCH(RG_K_RMSNORM, launch_rmsnorm(pol->dtype, pol->x, pol->g_attn[0], pol->d, pol->cfg.rms_eps, pol->abuf,
                                       pol->a_plane, nullptr, pol->state, rows_ub, st));
  if ((rc = run_layers(pol, st, pol->state, rows_ub, ctx_max, true, pre))) return rc;
  if ((rc = run_head(pol, st, pol->state, rows_ub, nullptr))) return rc;
  LAUNCH(RG_K_SAMPLE, launch_sample(sm, rows_ub, st));
  LAUNCH(RG_K_COMPACT, launch_compact(ca, st));
  return RG_OK;
}

// A decode-step graph per row bucket, captured on first use in a rollout.
struct StepGraphs {
  std::vector<std::pair<int, hipGraphExec_t>> execs;
  hipStream_t launched_on = nullptr;   // set once a graph has been launched
  ~StepGraphs() {
    // an early error return may leave replays in flight: let them finish first
    if (launched_on) (void)hipStreamSynchronize(launched_on);
    for (auto& g : execs) (void)hipGraphExecDestroy(g.second);
  }
};

int step_graph(rg_policy* pol, StepGraphs& gs, int rows_ub, int ctx_max, const SampleArgs& sm,
               const CompactArgs& ca, const PrefixPass* pre, hipGraphExec_t* out) {
  for (auto& g : gs.execs)
    if (g.first == rows_ub) { *out = g.second; return RG_OK; }
  HIPTRY(hipStreamBeginCapture(pol->cap_st, hipStreamCaptureModeThreadLocal));
  const int rc = enqueue_step(pol, pol->cap_st, rows_ub, ctx_max, sm, ca, pre);
  hipGraph_t graph = nullptr;
  const hipError_t e = hipStreamEndCapture(pol->cap_st, &graph);
  if (rc) {
    if (graph) (void)hipGraphDestroy(graph);
    return rc;
  }
  if (e != hipSuccess) return fail(RG_EHIP, std::string("hipStreamEndCapture: ") + hipGetErrorString(e));
  hipGraphExec_t exec = nullptr;
  const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (ei != hipSuccess) return fail(RG_EHIP, std::string("hipGraphInstantiate: ") + hipGetErrorString(ei));
  gs.execs.emplace_back(rows_ub, exec);
  *out = exec;
  return RG_OK;
}

// Prompts and group sizes of one call, checked against the policy's limits.
struct GroupRun {
  int P = 0, N = 0, max_plen = 0, T_pre = 0;
};

int check_groups(const rg_policy* pol, const char* who, const int32_t* prompt_len, int32_t P, const int32_t* G,
                 int32_t max_new, GroupRun* gr) {
  const rg_limits& lim = pol->lim;
  const std::string w(who);
  if (P < 1) return fail(RG_EINVAL, w + ": P < 1");
  if (max_new < 1) return fail(RG_EINVAL, w + ": max_new < 1");
  if (P > lim.max_prompts) return fail(RG_ENOMEM, w + ": P exceeds limits.max_prompts");
  int64_t N = 0, T_pre = 0, pre_pages = 0;
  int max_plen = 0;
  for (int p = 0; p < P; ++p) {
    if (prompt_len[p] < 1) return fail(RG_EINVAL, w + ": prompt_len < 1");
    if (G[p] < 1) return fail(RG_EINVAL, w + ": G < 1");
    N += G[p];
    T_pre += prompt_len[p];
    max_plen = std::max(max_plen, prompt_len[p]);
    pre_pages += ceil_div(prompt_len[p], pol->page_tok);
  }
  if (N > lim.max_seqs) return fail(RG_ENOMEM, w + ": sum(G) exceeds limits.max_seqs");
  if (T_pre > lim.max_prompt_tokens) return fail(RG_ENOMEM, w + ": prompt tokens exceed limits");
  if ((int64_t)max_plen + max_new > lim.max_context) return fail(RG_ENOMEM, w + ": context exceeds limits");
  if (pre_pages > pol->pool_pages) return fail(RG_ENOMEM, w + ": prompt pages exceed the KV pool");
  gr->P = P; gr->N = (int)N; gr->max_plen = max_plen; gr->T_pre = (int)T_pre;
  return RG_OK;
}

// Copies prompt lengths, G and (when given) per-sequence forced lengths into
// device memory through the pinned staging buffer.
int stage_groups(rg_policy* pol, hipStream_t st, const GroupRun& gr, const int32_t* prompt_len, const int32_t* G,
                 const int32_t* forced_len) {
  int32_t* hs = pol->h_stage;
  HIPTRY(hipStreamSynchronize(st));   // the staging buffer may still feed an earlier call's copies
  std::memcpy(hs, prompt_len, (size_t)gr.P * 4);
  std::memcpy(hs + gr.P, G, (size_t)gr.P * 4);
  HIPTRY(hipMemcpyAsync(pol->plen, hs, (size_t)gr.P * 4, hipMemcpyHostToDevice, st));
  HIPTRY(hipMemcpyAsync(pol->G_dev, hs + gr.P, (size_t)gr.P * 4, hipMemcpyHostToDevice, st));
  if (forced_len) {
    std::memcpy(hs + 2 * gr.P, forced_len, (size_t)gr.N * 4);
    HIPTRY(hipMemcpyAsync(pol->seq_forced, hs + 2 * gr.P, (size_t)gr.N * 4, hipMemcpyHostToDevice, st));
  }
  return RG_OK;
}

// Set-up (offsets, prompt page tables, free stack, output padding), the
// prefill of every prompt (pol->logits then holds each prompt's
// last-position logits) and the sibling fork with its copy-on-write pages.
// tokens_out may be NULL (left untouched).
int prefill_and_fork(rg_policy* pol, hipStream_t st, const GroupRun& gr, const int32_t* prompts,
                     const int32_t* prompt_len, const int32_t* G, int32_t max_new, bool share, int32_t* tokens_out,
                     float* logprobs_out) {
  const int P = gr.P, N = gr.N;
  SetupArgs sa{};
  sa.P = P; sa.n_seq = N; sa.max_new = max_new; sa.page_tok = pol->page_tok; sa.max_pages = pol->max_pages;
  sa.pool_pages = pol->pool_pages; sa.plen = pol->plen; sa.prompt_off = pol->prompt_off; sa.grp_off = pol->grp_off;
  sa.G = pol->G_dev; sa.page_tab = pol->page_tab; sa.free_stack = pol->free_stack; sa.state = pol->state;
  sa.tokens_out = tokens_out; sa.logprobs_out = logprobs_out; sa.last_rows = pol->last_rows;
  LAUNCH(RG_K_SETUP, launch_setup(sa, st));

  const int* d_pre = pol->state + 5;
  LAUNCH(RG_K_SETUP, launch_prefill_rows(pol->prompt_off, P, N, pol->row_tab, pol->row_pos, pol->row_beg, gr.T_pre,
                                         st));
  LAUNCH(RG_K_EMBED, launch_embed(pol->dtype, pol->w_embed, pol->d, pol->V, prompts, pol->x, pol->state + 7, d_pre,
                                  gr.T_pre, st));
  LAUNCH(RG_K_RMSNORM, launch_rmsnorm(pol->dtype, pol->x, pol->g_attn[0], pol->d, pol->cfg.rms_eps, pol->abuf,
                                       pol->a_plane, nullptr, d_pre, gr.T_pre, st));
  int rc = run_layers(pol, st, d_pre, gr.T_pre, gr.max_plen, false, nullptr);
  if (rc) return rc;
  if ((rc = run_head(pol, st, pol->state + 6, P, pol->last_rows))) return rc;

  ForkArgs fa{};
  fa.P = P; fa.n_seq = N; fa.page_tok = pol->page_tok; fa.max_pages = pol->max_pages;
  fa.share = share ? 1 : 0;
  fa.grp_off = pol->grp_off; fa.plen = pol->plen; fa.page_tab = pol->page_tab; fa.seq_grp = pol->seq_grp;
  fa.seq_npages = pol->seq_npages; fa.seq_nshared = pol->seq_nshared; fa.act_seq = pol->act_seq;
  fa.free_stack = pol->free_stack; fa.state = pol->state; fa.copy_pairs = pol->copy_pairs;
  LAUNCH(RG_K_SETUP, launch_fork(fa, st));
  int max_pairs = 0;
  for (int p = 0; p < P; ++p) {
    const int n_pref = (int)ceil_div(prompt_len[p], pol->page_tok);
    const int need = share ? (prompt_len[p] % pol->page_tok ? 1 : 0) : n_pref;
    max_pairs += need * G[p];
  }
  LAUNCH(RG_K_SETUP, launch_page_copy(pol->dtype, pol->kv_pool, pol->geom, pol->copy_pairs, max_pairs,
                                      pol->state, st));
  return RG_OK;
}

// Profiling state of a call that takes RG_FLAG_PROFILE.
int prof_begin(rg_policy* pol, bool on, uint32_t kinds) {
  pol->prof = on;
  pol->prof_mask = kinds ? kinds : 0xFFFFFFFFu;
  if (pol->prof) {
    if (pol->prof_ev.empty()) {
      pol->prof_ev.resize(2 * RG_PROF_RING);
      pol->prof_kind.resize(RG_PROF_RING);
      pol->prof_ph.resize(RG_PROF_RING);
      for (auto& e : pol->prof_ev) HIPTRY(hipEventCreate(&e));
    }
    std::memset(pol->kt_ms, 0, sizeof(pol->kt_ms));
    std::memset(pol->kt_n, 0, sizeof(pol->kt_n));
    pol->prof_head = pol->prof_tail = 0;
  }
  pol->prof_phase = 0;
  return RG_OK;
}

int prof_end(rg_policy* pol) {
  int rc;
  if (pol->prof)
    while (pol->prof_tail < pol->prof_head)
      if ((rc = prof_drain_one(pol))) return rc;
  return RG_OK;
}

int copy_weight(rg_policy* pol, void* dst, const void* src, size_t bytes, const char* what) {
  if (!src) return fail(RG_EINVAL, std::string("weights: NULL ") + what);
  HIPTRY(hipMemcpy(dst, src, bytes, hipMemcpyDeviceToDevice));
  return RG_OK;
}

}  // namespace

// ====================================================================== C ABI
extern "C" {

const char* rg_last_error(void) { return g_err.c_str(); }

int rg_policy_create(const rg_config* cfg, const rg_weights* w, const rg_limits* limits, rg_policy** out) {
  if (!cfg || !w || !limits || !out) return fail(RG_EINVAL, "rg_policy_create: NULL argument");
  *out = nullptr;
  const rg_config c = *cfg;
  if (c.n_layers < 1 || c.d_model < 1 || c.n_q_heads < 1 || c.n_kv_heads < 1 || c.head_dim < 2 || c.ffn_dim < 1 ||
      c.vocab < 2 || c.eos_id < 0 || c.eos_id >= c.vocab || !(c.rope_theta > 0.f) || !(c.rms_eps >= 0.f))
    return fail(RG_EINVAL, "rg_policy_create: invalid config");
  if (c.dtype != RG_DTYPE_F32 && c.dtype != RG_DTYPE_BF16) return fail(RG_EUNSUPPORTED, "unsupported dtype");
  if (c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 128)
    return fail(RG_EUNSUPPORTED, "unsupported shape: head_dim must be 32, 64 or 128 (bf16 models: 64 or 128)");
  if (c.dtype == RG_DTYPE_BF16 && c.head_dim == 32)
    return fail(RG_EUNSUPPORTED, "unsupported shape: bf16 models need head_dim 64 or 128");
  if (c.head_dim % 8 || c.head_dim > 256 || c.n_q_heads % c.n_kv_heads || c.n_q_heads / c.n_kv_heads > 8 ||
      c.d_model % 64 || (c.n_q_heads * c.head_dim) % 64 || c.ffn_dim % 64 || c.vocab % 16)
    return fail(RG_EUNSUPPORTED, "unsupported shape: need head_dim%8==0, head_dim<=256, n_q/n_kv integer <= 8, "
                                 "d_model, n_q*head_dim, ffn_dim multiples of 64, vocab multiple of 16");
  const rg_limits lim = *limits;
  if (lim.max_seqs < 1 || lim.max_prompts < 1 || lim.max_prompt_tokens < 1 || lim.max_context < 2 ||
      lim.kv_pool_pages < 0)
    return fail(RG_EINVAL, "rg_policy_create: invalid limits");

  // Owned here until creation succeeds: every early return (HIPTRY included)
  // frees the policy and the device memory it holds so far.
  std::unique_ptr<rg_policy> owner(new rg_policy());
  rg_policy* pol = owner.get();
  auto bail = [](int rc) { return rc; };
  pol->cfg = c;
  pol->lim = lim;
  pol->dtype = c.dtype;
  pol->eb = c.dtype == RG_DTYPE_BF16 ? 2 : 4;
  pol->d = c.d_model; pol->V = c.vocab; pol->L = c.n_layers; pol->F = c.ffn_dim; pol->hd = c.head_dim;
  pol->nq = c.n_q_heads; pol->nkv = c.n_kv_heads;
  pol->q_dim = c.n_q_heads * c.head_dim;
  pol->kv_dim = c.n_kv_heads * c.head_dim;
  pol->qkv_n = pol->q_dim + 2 * pol->kv_dim;
  pol->max_pages = (int)ceil_div(lim.max_context, pol->page_tok) + 1;
  pol->m_act = std::max(lim.max_prompt_tokens, lim.max_seqs);
  KvGeom& g = pol->geom;
  g.page_tok = pol->page_tok; g.n_layers = pol->L; g.n_kv = pol->nkv; g.head_dim = pol->hd;
  g.slab_elems = 2LL * pol->nkv * pol->page_tok * pol->hd;
  const size_t eb = pol->eb;
  const int64_t d = pol->d;
  int rc;

  // ---- weights (repacked: [wq; wk; wv] and [w_gate; w_up] stacked by rows)
  if ((rc = pol->alloc(&pol->w_embed, (size_t)pol->V * d * eb))) return bail(rc);
  if ((rc = copy_weight(pol, pol->w_embed, w->embed, (size_t)pol->V * d * eb, "embed"))) return bail(rc);
  if ((rc = pol->alloc(&pol->w_lm, (size_t)pol->V * d * eb))) return bail(rc);
  if ((rc = copy_weight(pol, pol->w_lm, w->lm_head, (size_t)pol->V * d * eb, "lm_head"))) return bail(rc);
  if ((rc = pol->alloc((void**)&pol->w_final, d * 4))) return bail(rc);
  if ((rc = copy_weight(pol, pol->w_final, w->final_norm, d * 4, "final_norm"))) return bail(rc);
  if (!w->attn_norm || !w->wq || !w->wk || !w->wv || !w->wo || !w->ffn_norm || !w->w_gate || !w->w_up || !w->w_down)
    return bail(fail(RG_EINVAL, "weights: NULL per-layer array"));
  for (int l = 0; l < pol->L; ++l) {
    void *qkv, *o, *gu, *dn;
    float *ga, *gf;
    // [wq; wk; wv] with each head's rows reordered in 16-row tiles as dims
    // (0-15, hd/2..hd/2+15, 16-31, hd/2+16.., ...): a rotated pair (d, d + hd/2)
    // then sits in two adjacent 16-column tiles of the product
    if ((rc = pol->alloc(&qkv, (size_t)pol->qkv_n * d * eb))) return bail(rc);
    if (!w->wq[l] || !w->wk[l] || !w->wv[l]) return bail(fail(RG_EINVAL, "weights: NULL wq/wk/wv"));
    {
      const int hd = pol->hd, half = hd / 2;
      const size_t row = (size_t)d * eb;
      const void* src[3] = {w->wq[l], w->wk[l], w->wv[l]};
      const int heads[3] = {pol->nq, pol->nkv, pol->nkv};
      size_t base = 0;
      for (int part = 0; part < 3; ++part) {
        for (int t = 0; t < hd / 16; ++t) {   // packed tile t of every head
          const int d0 = (t & 1) ? half + (t >> 1) * 16 : (t >> 1) * 16;
          HIPTRY(hipMemcpy2D((char*)qkv + (base + (size_t)t * 16) * row, (size_t)hd * row,
                             (const char*)src[part] + (size_t)d0 * row, (size_t)hd * row, 16 * row, heads[part],
                             hipMemcpyDeviceToDevice));
        }
        base += (size_t)heads[part] * hd;
      }
    }
    if ((rc = pol->alloc(&o, (size_t)d * pol->q_dim * eb))) return bail(rc);
    if ((rc = copy_weight(pol, o, w->wo[l], (size_t)d * pol->q_dim * eb, "wo"))) return bail(rc);
    // gate/up interleaved in blocks of 16 rows: [gate 16b..16b+15 | up 16b..16b+15] for block b,
    // so one 32-column tile of the product holds both halves of 16 SwiGLU outputs
    if ((rc = pol->alloc(&gu, (size_t)2 * pol->F * d * eb))) return bail(rc);
    if (!w->w_gate[l] || !w->w_up[l]) return bail(fail(RG_EINVAL, "weights: NULL w_gate/w_up"));
    {
      const size_t blk = (size_t)16 * d * eb;
      HIPTRY(hipMemcpy2D(gu, 2 * blk, w->w_gate[l], blk, blk, pol->F / 16, hipMemcpyDeviceToDevice));
      HIPTRY(hipMemcpy2D((char*)gu + blk, 2 * blk, w->w_up[l], blk, blk, pol->F / 16, hipMemcpyDeviceToDevice));
    }
    if ((rc = pol->alloc(&dn, (size_t)d * pol->F * eb))) return bail(rc);
    if ((rc = copy_weight(pol, dn, w->w_down[l], (size_t)d * pol->F * eb, "w_down"))) return bail(rc);
    if ((rc = pol->alloc((void**)&ga, d * 4))) return bail(rc);
    if ((rc = copy_weight(pol, ga, w->attn_norm[l], d * 4, "attn_norm"))) return bail(rc);
    if ((rc = pol->alloc((void**)&gf, d * 4))) return bail(rc);
    if ((rc = copy_weight(pol, gf, w->ffn_norm[l], d * 4, "ffn_norm"))) return bail(rc);
    pol->w_qkv.push_back(qkv); pol->w_o.push_back(o); pol->w_gu.push_back(gu); pol->w_down.push_back(dn);
    pol->g_attn.push_back(ga); pol->g_ffn.push_back(gf);
  }

  // ---- RoPE table: angle pos * theta^(-2i/hd) in double, stored as fp32 cos/sin
  {
    const int half = pol->hd / 2;
    const size_t n = (size_t)lim.max_context * half;
    std::vector<float> cs(n), sn(n);
    for (int i = 0; i < half; ++i) {
      const double inv = std::pow((double)c.rope_theta, -2.0 * i / (double)pol->hd);
      for (int p = 0; p < lim.max_context; ++p) {
        const double a = (double)p * inv;
        cs[(size_t)p * half + i] = (float)std::cos(a);
        sn[(size_t)p * half + i] = (float)std::sin(a);
      }
    }
    if ((rc = pol->alloc((void**)&pol->rope_cos, n * 4))) return bail(rc);
    if ((rc = pol->alloc((void**)&pol->rope_sin, n * 4))) return bail(rc);
    HIPTRY(hipMemcpy(pol->rope_cos, cs.data(), n * 4, hipMemcpyHostToDevice));
    HIPTRY(hipMemcpy(pol->rope_sin, sn.data(), n * 4, hipMemcpyHostToDevice));
  }

  // ---- KV page pool
  pol->pool_pages = lim.kv_pool_pages;
  if (pol->pool_pages == 0)
    pol->pool_pages = ceil_div(lim.max_prompt_tokens, pol->page_tok) + lim.max_prompts +
                      (int64_t)lim.max_seqs * (ceil_div(lim.max_context, pol->page_tok) + 1);
  if (pol->pool_pages > INT32_MAX) return bail(fail(RG_ENOMEM, "KV pool exceeds 2^31 pages"));
  g.page_stride = g.slab_elems;                      // layer-major pool
  g.layer_stride = g.slab_elems * pol->pool_pages;
  if ((rc = pol->alloc(&pol->kv_pool, (size_t)pol->pool_pages * g.slab_elems * pol->L * eb))) return bail(rc);

  // ---- workspace
  const int64_t M = pol->m_act, S = lim.max_seqs, P = lim.max_prompts;
  // the rollout needs max(S, P) rows of logits; the recompute's lm head runs
  // in slices of this many rows, and slices above 1024 rows take the 256 x 256
  // projection tiles
  pol->logit_rows = std::max<int64_t>({S, P, std::min<int64_t>(M, RG_LM_SLICE_ROWS)});
  const int64_t maxN = std::max<int64_t>({pol->qkv_n, 2LL * pol->F, d});
  pol->cpart_elems = std::max(M * maxN, (int64_t)RG_SPLIT_MAX * S * maxN);
  // fp32 models run every projection through the partial buffer, the lm head
  // too: up to max(M, logit_rows) rows of the vocabulary
  if (pol->dtype != RG_DTYPE_BF16)
    pol->cpart_elems = std::max(pol->cpart_elems, std::max(M, pol->logit_rows) * (int64_t)pol->V);
  // (row, context chunk) slots of one attention launch: decode steps (rows <=
  // S, prefix slots and chunks), and a full activation chunk of prefill or
  // recompute rows, which splits contexts longer than one chunk's span
  pol->att_rowchunks = std::max<int64_t>(
      std::max<int64_t>(lim.max_prompt_tokens, S) + ATT_ITEMS_TARGET +
          S * (RG_PRE_MAX_SLOTS + ceil_div(lim.max_context, 1024)),
      M * att_row_chunks((int)std::min<int64_t>(M, INT32_MAX), pol->nkv, lim.max_context));
  pol->hist_cap = lim.max_context;
  struct Piece { void** p; size_t bytes; };
  const int64_t kmax = std::max<int64_t>({d, pol->q_dim, pol->F});
  pol->a_plane = pol->dtype == RG_DTYPE_BF16 ? M * kmax : 0;
  std::vector<Piece> pieces = {
      {(void**)&pol->x, (size_t)(M * d * 4)},
      {&pol->abuf, (size_t)(M * kmax * 4)},   // fp32, or two bf16 planes
      {&pol->abuf2, (size_t)(M * kmax * 4)},
      {(void**)&pol->cpart, (size_t)(pol->cpart_elems * 4)},
      {(void**)&pol->qbuf, (size_t)(M * pol->q_dim * 4)},
      {(void**)&pol->att_o, (size_t)(pol->att_rowchunks * pol->nq * pol->hd * 4)},
      {(void**)&pol->att_ml, (size_t)(pol->att_rowchunks * pol->nq * 2 * 4)},
      {(void**)&pol->logits, (size_t)(pol->logit_rows * pol->V * 4)},
      {(void**)&pol->sample_part, (size_t)(std::max(S, P) * RG_SAMPLE_SLICES_MAX * 4 * 4)},
      {(void**)&pol->page_tab, (size_t)((S + P) * pol->max_pages * 4)},
      {(void**)&pol->seq_grp, (size_t)(S * 4)},
      {(void**)&pol->seq_npages, (size_t)(S * 4)},
      {(void**)&pol->seq_nshared, (size_t)(S * 4)},
      {(void**)&pol->seq_forced, (size_t)(S * 4)},
      {(void**)&pol->grp_off, (size_t)((P + 1) * 4)},
      {(void**)&pol->prompt_off, (size_t)((P + 1) * 4)},
      {(void**)&pol->plen, (size_t)(P * 4)},
      {(void**)&pol->G_dev, (size_t)(P * 4)},
      {(void**)&pol->last_rows, (size_t)(P * 4)},
      {(void**)&pol->act_seq, (size_t)(S * 4)},
      {(void**)&pol->act_tok, (size_t)(S * 4)},
      {(void**)&pol->done, (size_t)(S * 4)},
      {(void**)&pol->row_tab, (size_t)(M * 4)},
      {(void**)&pol->row_pos, (size_t)(M * 4)},
      {(void**)&pol->row_beg, (size_t)(M * 4)},
      {(void**)&pol->grp_row0, (size_t)(P * 4)},
      {(void**)&pol->grp_row1, (size_t)(P * 4)},
      {(void**)&pol->coff, (size_t)((S + 1) * 4)},
      {(void**)&pol->row_tgt, (size_t)(M * 4)},
      {(void**)&pol->row_out, (size_t)(M * 4)},
      {(void**)&pol->row_lrow, (size_t)(S * 4)},
      {(void**)&pol->tile_r0, (size_t)((M + S + 1) * 4)},
      {(void**)&pol->tile_nr, (size_t)((M + S + 1) * 4)},
      {(void**)&pol->free_stack, (size_t)(pol->pool_pages * 4)},
      {(void**)&pol->state, 64},
      {(void**)&pol->copy_pairs, (size_t)(2 * S * pol->max_pages * 4)},
      {(void**)&pol->hist_active, (size_t)(pol->hist_cap * 4)},
      {(void**)&pol->hist_groups, (size_t)(pol->hist_cap * 4)},
      {(void**)&pol->hist_ctx, (size_t)(pol->hist_cap * 8)},
  };
  size_t total = 0;
  for (auto& pc : pieces) total += (pc.bytes + 255) & ~(size_t)255;
  char* arena;
  if ((rc = pol->alloc((void**)&arena, total))) return bail(rc);
  for (auto& pc : pieces) {
    *pc.p = arena;
    arena += (pc.bytes + 255) & ~(size_t)255;
  }
  {
    hipError_t e = hipHostMalloc((void**)&pol->h_stage, (size_t)(2 * P + S + 64) * 4, hipHostMallocDefault);
    if (e != hipSuccess) return bail(fail(RG_EHIP, std::string("hipHostMalloc: ") + hipGetErrorString(e)));
    e = hipHostMalloc((void**)&pol->h_ring, (size_t)RG_RING * 8 * 4, hipHostMallocDefault);
    if (e != hipSuccess) return bail(fail(RG_EHIP, std::string("hipHostMalloc: ") + hipGetErrorString(e)));
    for (auto& ev : pol->ring_ev) {
      e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
      if (e != hipSuccess) return bail(fail(RG_EHIP, std::string("hipEventCreate: ") + hipGetErrorString(e)));
    }
    for (auto& ev : pol->phase_ev) {
      e = hipEventCreate(&ev);
      if (e != hipSuccess) return bail(fail(RG_EHIP, std::string("hipEventCreate: ") + hipGetErrorString(e)));
    }
    e = hipStreamCreateWithFlags(&pol->cap_st, hipStreamNonBlocking);
    if (e != hipSuccess) return bail(fail(RG_EHIP, std::string("hipStreamCreate: ") + hipGetErrorString(e)));
    const char* env = getenv("RG_NO_GRAPHS");
    pol->use_graphs = !(env && env[0] == '1');
    const char* pe = getenv("RG_PROGRESS");
    pol->progress_every = pe ? std::max(0, atoi(pe)) : 0;
  }
  *out = owner.release();
  return RG_OK;
}

void rg_policy_destroy(rg_policy* pol) { delete pol; }

int64_t rg_policy_device_bytes(const rg_policy* pol) { return pol ? pol->dev_bytes : 0; }

int rollout_group(rg_policy* pol, const int32_t* prompts, const int32_t* prompt_len, int32_t P, const int32_t* G,
                  int32_t max_new, uint64_t seed, const rg_sampling* opts, int32_t* tokens, int32_t* lengths,
                  float* logprobs, void* stream) {
  if (!pol || !prompts || !prompt_len || !G || !tokens || !lengths || !logprobs)
    return fail(RG_EINVAL, "rollout_group: NULL argument");
  hipStream_t st = (hipStream_t)stream;
  GroupRun gr;
  int rc = check_groups(pol, "rollout_group", prompt_len, P, G, max_new, &gr);
  if (rc) return rc;
  const int64_t N = gr.N;
  const int max_plen = gr.max_plen;
  rg_sampling o{};
  o.temperature = 1.f;
  if (opts) o = *opts;
  if (!(o.temperature > 0.f) || !std::isfinite(o.temperature)) return fail(RG_EINVAL, "rollout_group: temperature <= 0");
  if (o.dump_steps < 0) return fail(RG_EINVAL, "rollout_group: dump_steps < 0");
  if (o.forced_len)
    for (int64_t s = 0; s < N; ++s)
      if (o.forced_len[s] < 1 || o.forced_len[s] > max_new) return fail(RG_EINVAL, "rollout_group: forced_len out of [1, max_new]");
  const int Ni = (int)N;

  if ((rc = prof_begin(pol, (o.flags & RG_FLAG_PROFILE) != 0, o.profile_kinds))) return rc;
  if ((rc = stage_groups(pol, st, gr, prompt_len, G, o.forced_len))) return rc;
  const int32_t* forced_dev = o.forced_len ? pol->seq_forced : nullptr;
  pol->phase_valid = false;
  HIPTRY(hipEventRecord(pol->phase_ev[0], st));
  if ((rc = prefill_and_fork(pol, st, gr, prompts, prompt_len, G, max_new, !(o.flags & RG_FLAG_NO_PREFIX_SHARING),
                             tokens, logprobs)))
    return rc;
  HIPTRY(hipEventRecord(pol->phase_ev[1], st));

  // ---- sampling / retirement of one step
  SampleArgs sm{};
  sm.V = pol->V; sm.eos = pol->cfg.eos_id; sm.max_new = max_new; sm.seed = seed; sm.temperature = o.temperature;
  sm.act_seq = pol->act_seq; sm.seq_grp = pol->seq_grp; sm.forced_len = forced_dev; sm.force_tokens = o.force_tokens;
  sm.dump_logits = o.dump_logits; sm.dump_steps = o.dump_steps; sm.n_seq = Ni; sm.tokens_out = tokens;
  sm.logprobs_out = logprobs; sm.next_tok = pol->act_tok; sm.done = pol->done; sm.d_rows = pol->state;
  sm.bad_token = pol->state + 7;
  sm.logits = pol->logits;
  sm.d_t = pol->state + 8;
  CompactArgs ca{};
  ca.max_new = max_new; ca.page_tok = pol->page_tok; ca.max_pages = pol->max_pages; ca.n_seq = Ni;
  ca.act_seq = pol->act_seq; ca.act_tok = pol->act_tok; ca.done = pol->done; ca.seq_grp = pol->seq_grp;
  ca.plen = pol->plen; ca.page_tab = pol->page_tab; ca.seq_npages = pol->seq_npages; ca.seq_nshared = pol->seq_nshared;
  ca.free_stack = pol->free_stack; ca.state = pol->state; ca.lengths = lengths; ca.hist_active = pol->hist_active;
  ca.hist_groups = pol->hist_groups; ca.hist_ctx = pol->hist_ctx; ca.hist_cap = pol->hist_cap;
  ca.P = P; ca.grp_row0 = pol->grp_row0; ca.grp_row1 = pol->grp_row1;

  // shared-prefix attention pass of the decode steps
  PrefixPass pp{};
  pp.P = P;
  pp.tab_base = Ni;
  for (int p = 0; p < P; ++p) {
    pp.max_group_rows = std::max(pp.max_group_rows, G[p]);
    pp.max_pref = std::max(pp.max_pref, prompt_len[p] / pol->page_tok * pol->page_tok);
  }
  const PrefixPass* pre =
      pol->dtype == RG_DTYPE_BF16 && (o.flags & RG_FLAG_GROUP_PREFIX) && pp.max_pref > 0 ? &pp : nullptr;

  auto snapshot = [&](int t) -> int {
    const int slot = t % RG_RING;
    HIPTRY(hipMemcpyAsync(pol->h_ring + 8 * slot, pol->state, 8 * sizeof(int32_t), hipMemcpyDeviceToHost, st));
    HIPTRY(hipEventRecord(pol->ring_ev[slot], st));
    return RG_OK;
  };

  // step 0: every sibling samples from its prompt's logits
  pol->prof_phase = 1;
  sm.logits_by_group = 1;
  sm.part = pol->sample_part;
  sm.n_slices = sample_slices(Ni);
  LAUNCH(RG_K_SAMPLE, launch_sample(sm, Ni, st));
  LAUNCH(RG_K_COMPACT, launch_compact(ca, st));
  if ((rc = snapshot(0))) return rc;
  HIPTRY(hipEventSynchronize(pol->ring_ev[0]));
  int known_t = 0, last_t = 0;
  int m_ub = pol->h_ring[0];
  bool oom = pol->h_ring[2] != 0;
  int n_steps = m_ub == 0 ? 1 : 0;

  // steps t >= 1, as captured graphs (one per row bucket) or, when kernels
  // are being timed, as direct launches; both run the same kernels with the
  // same arguments.  The attention chunk plan covers the longest possible
  // context, so it does not change from step to step.
  sm.logits_by_group = 0;
  const int ctx_all = max_plen + max_new;
  StepGraphs graphs;
  const bool graphs_on = pol->use_graphs && !pol->prof;
  for (int t = 1; t < max_new && n_steps == 0 && !oom; ++t) {
    // refresh the upper bound from completed snapshots; never run too far ahead
    while (known_t + 1 < t) {
      const int nx = (known_t + 1) % RG_RING;
      if (t - known_t > RG_LOOKAHEAD) HIPTRY(hipEventSynchronize(pol->ring_ev[nx]));
      else if (hipEventQuery(pol->ring_ev[nx]) != hipSuccess) break;
      ++known_t;
      m_ub = pol->h_ring[8 * nx];
      if (pol->h_ring[8 * nx + 2]) oom = true;
      if (m_ub == 0) { n_steps = known_t + 1; break; }
    }
    if (n_steps || oom) break;
    const int rows_ub = std::min(row_bucket(m_ub), pol->m_act);
    if (graphs_on) {
      hipGraphExec_t exec;
      if ((rc = step_graph(pol, graphs, rows_ub, ctx_all, sm, ca, pre, &exec))) return rc;
      graphs.launched_on = st;
      HIPTRY(hipGraphLaunch(exec, st));
    } else {
      pol->prof_phase = bucket_phase(rows_ub);
      if ((rc = enqueue_step(pol, st, rows_ub, ctx_all, sm, ca, pre))) return rc;
    }
    if ((rc = snapshot(t))) return rc;
    last_t = t;
    if (pol->progress_every && t % pol->progress_every == 0) {
      fprintf(stderr, "# decode step %d enqueued; step %d done with %d active rows\n", t, known_t, m_ub);
      fflush(stderr);
    }
  }
  HIPTRY(hipEventRecord(pol->phase_ev[2], st));
  HIPTRY(hipStreamSynchronize(st));
  pol->phase_valid = true;
  // snapshots the loop has not read yet (at most RG_LOOKAHEAD of them)
  for (int k = known_t + 1; k <= last_t; ++k) {
    const int nx = k % RG_RING;
    if (pol->h_ring[8 * nx + 2]) oom = true;
    if (pol->h_ring[8 * nx] == 0 && n_steps == 0) n_steps = k + 1;
  }
  if (n_steps == 0) n_steps = last_t + 1;
  const bool bad_token = pol->h_ring[8 * (last_t % RG_RING) + 7] != 0;
  pol->last_steps = n_steps;
  if ((rc = prof_end(pol))) return rc;
  if (oom) return fail(RG_ENOMEM, "rollout_group: the KV page pool ran out");
  if (bad_token) return fail(RG_EINVAL, "rollout_group: a prompt or forced token id is outside [0, vocab)");
  return RG_OK;
}

int recompute_logprobs(rg_policy* pol, const int32_t* prompts, const int32_t* prompt_len, int32_t P, const int32_t* G,
                       const int32_t* tokens, const int32_t* lengths, int32_t max_new, float temperature, int32_t flags,
                       float* logprobs, void* stream) {
  if (!pol || !prompts || !prompt_len || !G || !tokens || !lengths || !logprobs)
    return fail(RG_EINVAL, "recompute_logprobs: NULL argument");
  hipStream_t st = (hipStream_t)stream;
  GroupRun gr;
  int rc = check_groups(pol, "recompute_logprobs", prompt_len, P, G, max_new, &gr);
  if (rc) return rc;
  if (!(temperature > 0.f) || !std::isfinite(temperature))
    return fail(RG_EINVAL, "recompute_logprobs: temperature <= 0");
  if ((int64_t)gr.N * max_new >= INT32_MAX) return fail(RG_EINVAL, "recompute_logprobs: N * max_new >= 2^31");
  const int N = gr.N;
  if ((rc = prof_begin(pol, (flags & RG_FLAG_PROFILE) != 0, 0))) return rc;
  if ((rc = stage_groups(pol, st, gr, prompt_len, G, nullptr))) return rc;
  if ((rc = prefill_and_fork(pol, st, gr, prompts, prompt_len, G, max_new, !(flags & RG_FLAG_NO_PREFIX_SHARING),
                             nullptr, logprobs)))
    return rc;

  // y_0 of every sequence, scored by its prompt's last-position logits
  pol->prof_phase = 1;
  LAUNCH(RG_K_SETUP, launch_first_rows(tokens, pol->seq_grp, N, max_new, pol->V, pol->row_lrow, pol->row_tgt,
                                       pol->row_out, pol->state + 7, st));
  LAUNCH(RG_K_LOGPROB, launch_token_logprob(pol->logits, pol->V, temperature, pol->row_lrow, pol->row_tgt,
                                            pol->row_out, logprobs, N, st));
  // pages for every completion position, and the row offsets
  ReserveArgs ra{};
  ra.n_seq = N; ra.max_new = max_new; ra.page_tok = pol->page_tok; ra.max_pages = pol->max_pages;
  ra.lengths = lengths; ra.plen = pol->plen; ra.seq_grp = pol->seq_grp; ra.seq_npages = pol->seq_npages;
  ra.page_tab = pol->page_tab; ra.free_stack = pol->free_stack; ra.coff = pol->coff; ra.state = pol->state;
  LAUNCH(RG_K_SETUP, launch_reserve(ra, st));
  HIPTRY(hipMemcpyAsync(pol->h_ring, pol->state, 16 * sizeof(int32_t), hipMemcpyDeviceToHost, st));
  HIPTRY(hipStreamSynchronize(st));
  if (pol->h_ring[2]) return fail(RG_ENOMEM, "recompute_logprobs: the KV page pool ran out");
  if (pol->h_ring[10]) return fail(RG_EINVAL, "recompute_logprobs: a length is outside [1, max_new]");
  const int64_t R = pol->h_ring[9];

  // the teacher-forced rows in chunks of m_act; the lm head in slices of the
  // logits buffer's rows
  const int chunk = pol->m_act;
  const int slice = (int)pol->logit_rows;
  const int ctx_all = gr.max_plen + max_new;
  const size_t row_bytes = (size_t)pol->d * pol->eb;
  int* d_chunk = pol->state + 11;
  int* d_slice = pol->state + 12;
  int* d_tiles = pol->state + 13;
  // bf16 models: attention by row tiles (32 positions of a sequence, 16 when
  // more than 6 query heads share a kv head, share each staged K/V block);
  // RG_FLAG_NO_ROW_TILES keeps the per-row pass
  const bool use_tiles = pol->dtype == RG_DTYPE_BF16 && !(flags & RG_FLAG_NO_ROW_TILES) &&
                         pol->nq / pol->nkv <= 8 && ctx_all <= 16384;
  const int tile_rows = att_tile_rows(pol->nq, pol->nkv);
  RecomputeRows rr{};
  rr.n_seq = N; rr.max_new = max_new; rr.V = pol->V; rr.d = pol->d; rr.coff = pol->coff; rr.tokens = tokens;
  rr.plen = pol->plen; rr.seq_grp = pol->seq_grp; rr.row_tab = pol->row_tab; rr.row_pos = pol->row_pos;
  rr.row_beg = pol->row_beg; rr.row_tgt = pol->row_tgt; rr.row_out = pol->row_out; rr.x = pol->x;
  rr.bad_token = pol->state + 7;
  GemmEpi store{};
  store.mode = GEMM_EPI_STORE; store.C = pol->logits; store.ldc = pol->V;
  for (int64_t r0 = 0; r0 < R; r0 += chunk) {
    const int n = (int)std::min<int64_t>(chunk, R - r0);
    rr.row0 = (int)r0;
    LAUNCH(RG_K_EMBED, launch_recompute_rows(pol->dtype, pol->w_embed, rr, n, st));
    LAUNCH(RG_K_SETUP, launch_fill_i32(d_chunk, 1, n, st));
    LAUNCH(RG_K_RMSNORM, launch_rmsnorm(pol->dtype, pol->x, pol->g_attn[0], pol->d, pol->cfg.rms_eps, pol->abuf,
                                         pol->a_plane, nullptr, d_chunk, n, st));
    RowTiles rt{d_tiles, (int)ceil_div(n, tile_rows) + std::min(n, N)};
    if (use_tiles) LAUNCH(RG_K_SETUP, launch_row_tiles(pol->row_tab, pol->coff, (int)r0, n, tile_rows, pol->tile_r0,
                                                       pol->tile_nr, d_tiles, st));
    if ((rc = run_layers(pol, st, d_chunk, n, ctx_all, true, nullptr, use_tiles ? &rt : nullptr))) return rc;
    for (int h0 = 0; h0 < n; h0 += slice) {
      const int m = std::min(slice, n - h0);
      LAUNCH(RG_K_SETUP, launch_fill_i32(d_slice, 1, m, st));
      if ((rc = gemm(pol, st, RG_K_GEMM_LM, (const char*)pol->abuf + (size_t)h0 * row_bytes, pol->d, pol->w_lm,
                     pol->V, d_slice, m, store, false)))
        return rc;
      LAUNCH(RG_K_LOGPROB, launch_token_logprob(pol->logits, pol->V, temperature, nullptr, pol->row_tgt + h0,
                                                pol->row_out + h0, logprobs, m, st));
    }
  }
  HIPTRY(hipMemcpyAsync(pol->h_ring, pol->state, 16 * sizeof(int32_t), hipMemcpyDeviceToHost, st));
  HIPTRY(hipStreamSynchronize(st));
  if ((rc = prof_end(pol))) return rc;
  if (pol->h_ring[7]) return fail(RG_EINVAL, "recompute_logprobs: a prompt or completion token id is outside [0, vocab)");
  return RG_OK;
}

namespace {
// Arguments of the clipped surrogate, checked on the host.
int surrogate_args(const char* who, const float* new_lp, const float* old_lp, const float* adv,
                   const int32_t* lengths, const int32_t* G, int32_t P, int32_t N, int32_t max_new,
                   const int32_t* keep, double eps_lo, double eps_hi, int32_t mode, double* out, SurrogateArgs* sa) {
  const std::string w(who);
  if (!new_lp || !old_lp || !adv || !lengths || !G || !out) return fail(RG_EINVAL, w + ": NULL argument");
  if (P < 1 || N < 1 || max_new < 1) return fail(RG_EINVAL, w + ": P, N and max_new must be >= 1");
  if (!(eps_lo >= 0.0 && eps_lo < 1.0) || !(eps_hi >= 0.0) || !std::isfinite(eps_hi))
    return fail(RG_EINVAL, w + ": need 0 <= eps_lo < 1 and 0 <= eps_hi");
  if (mode != RG_LOSS_TOKEN_MEAN && mode != RG_LOSS_SEQ_MEAN) return fail(RG_EINVAL, w + ": unknown mode");
  *sa = SurrogateArgs{};
  sa->new_lp = new_lp; sa->old_lp = old_lp; sa->adv = adv; sa->lengths = lengths; sa->G = G; sa->keep = keep;
  sa->P = P; sa->N = N; sa->max_new = max_new; sa->mode = mode; sa->eps_lo = eps_lo; sa->eps_hi = eps_hi;
  sa->out = out;
  return RG_OK;
}
}  // namespace

int grpo_surrogate(const float* new_lp, const float* old_lp, const float* adv, const int32_t* lengths,
                   const int32_t* G, int32_t P, int32_t N, int32_t max_new, const int32_t* keep, double eps_lo,
                   double eps_hi, int32_t mode, double* out, void* stream) {
  SurrogateArgs sa;
  int rc = surrogate_args("grpo_surrogate", new_lp, old_lp, adv, lengths, G, P, N, max_new, keep, eps_lo, eps_hi,
                          mode, out, &sa);
  if (rc) return rc;
  // per-sequence records: stream-ordered scratch of this call alone
  hipStream_t st = (hipStream_t)stream;
  SurrogateRec* rec = nullptr;
  HIPTRY(hipMallocAsync((void**)&rec, (size_t)N * sizeof(SurrogateRec), st));
  const hipError_t e = launch_surrogate(sa, rec, st);
  const hipError_t ef = hipFreeAsync(rec, st);
  if (e != hipSuccess) return fail(RG_EHIP, std::string("grpo_surrogate launch: ") + hipGetErrorString(e));
  if (ef != hipSuccess) return fail(RG_EHIP, std::string("grpo_surrogate hipFreeAsync: ") + hipGetErrorString(ef));
  return RG_OK;
}

int grpo_surrogate_noalloc(const float* new_lp, const float* old_lp, const float* adv, const int32_t* lengths,
                           const int32_t* G, int32_t P, int32_t N, int32_t max_new, const int32_t* keep,
                           double eps_lo, double eps_hi, int32_t mode, double* out, void* stream) {
  SurrogateArgs sa;
  int rc = surrogate_args("grpo_surrogate_noalloc", new_lp, old_lp, adv, lengths, G, P, N, max_new, keep, eps_lo,
                          eps_hi, mode, out, &sa);
  if (rc) return rc;
  if (N > SURROGATE_NOALLOC_MAX_SEQS)
    return fail(RG_EINVAL, "grpo_surrogate_noalloc: N exceeds the static scratch (" +
                               std::to_string(SURROGATE_NOALLOC_MAX_SEQS) + " sequences)");
  SurrogateRec* rec = nullptr;
  hipError_t e = surrogate_static_scratch(&rec);
  if (e != hipSuccess) return fail(RG_EHIP, std::string("grpo_surrogate_noalloc scratch: ") + hipGetErrorString(e));
  e = launch_surrogate(sa, rec, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RG_EHIP, std::string("grpo_surrogate_noalloc launch: ") + hipGetErrorString(e));
  return RG_OK;
}

int group_advantage(const float* rewards, const int32_t* G, int32_t P, int32_t N, float eps, int32_t ddof, float* adv,
                    void* stream) {
  if (!rewards || !G || !adv) return fail(RG_EINVAL, "group_advantage: NULL argument");
  if (P < 1 || N < 1) return fail(RG_EINVAL, "group_advantage: P < 1 or N < 1");
  if (!(eps >= 0.f)) return fail(RG_EINVAL, "group_advantage: eps < 0");
  if (ddof != 0 && ddof != 1) return fail(RG_EINVAL, "group_advantage: ddof must be 0 or 1");
  if ((const void*)rewards == (const void*)adv) return fail(RG_EINVAL, "group_advantage: adv aliases rewards");
  hipError_t e = launch_group_advantage(rewards, G, P, N, eps, ddof, adv, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RG_EHIP, std::string("group_advantage launch: ") + hipGetErrorString(e));
  return RG_OK;
}

int group_filter(const float* rewards, const int32_t* G, int32_t P, int32_t N, int32_t* keep, int32_t* kept_ids,
                 int32_t* n_kept, void* stream) {
  if (!rewards || !G || !keep || !kept_ids || !n_kept) return fail(RG_EINVAL, "group_filter: NULL argument");
  if (P < 1 || N < 1) return fail(RG_EINVAL, "group_filter: P < 1 or N < 1");
  hipError_t e = launch_group_filter(rewards, G, P, N, keep, kept_ids, n_kept, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RG_EHIP, std::string("group_filter launch: ") + hipGetErrorString(e));
  return RG_OK;
}

int rg_philox_blocks(uint64_t key0, uint64_t key1, const uint64_t* ctr, int64_t n, uint64_t* out, void* stream) {
  if (!ctr || !out || n < 0) return fail(RG_EINVAL, "rg_philox_blocks: bad argument");
  hipError_t e = launch_philox_blocks(key0, key1, ctr, n, out, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RG_EHIP, std::string("rg_philox_blocks: ") + hipGetErrorString(e));
  return RG_OK;
}

int rg_gumbel_bits(uint64_t seed, int32_t t, int32_t s, int32_t vocab, uint32_t* out, void* stream) {
  if (!out || vocab < 1 || t < 0 || s < 0) return fail(RG_EINVAL, "rg_gumbel_bits: bad argument");
  hipError_t e = launch_gumbel_bits(seed, t, s, vocab, out, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RG_EHIP, std::string("rg_gumbel_bits: ") + hipGetErrorString(e));
  return RG_OK;
}

int rg_hbm_probe(const void* src, void* dst, int64_t bytes, int32_t mode, int32_t blocks, void* stream) {
  if (!src || !dst || bytes < 16 || bytes % 16 || (mode != 0 && mode != 1) || blocks < 1 || blocks > (1 << 20))
    return fail(RG_EINVAL, "rg_hbm_probe: bad argument");
  hipError_t e = launch_hbm_probe(src, dst, bytes, mode, blocks, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RG_EHIP, std::string("rg_hbm_probe: ") + hipGetErrorString(e));
  return RG_OK;
}

int rg_step_history(const rg_policy* pol, int32_t cap, int32_t* n_steps, int32_t* active, int32_t* groups,
                    int64_t* ctx) {
  if (!pol || cap < 0) return fail(RG_EINVAL, "rg_step_history: bad argument");
  if (n_steps) *n_steps = pol->last_steps;
  const int n = std::min(cap, std::min(pol->last_steps, pol->hist_cap));
  if (n <= 0) return RG_OK;
  if (active) HIPTRY(hipMemcpy(active, pol->hist_active, (size_t)n * 4, hipMemcpyDeviceToHost));
  if (groups) HIPTRY(hipMemcpy(groups, pol->hist_groups, (size_t)n * 4, hipMemcpyDeviceToHost));
  if (ctx) HIPTRY(hipMemcpy(ctx, pol->hist_ctx, (size_t)n * 8, hipMemcpyDeviceToHost));
  return RG_OK;
}

int rg_phase_times(const rg_policy* pol, double* prefill_ms, double* decode_ms) {
  if (!pol) return fail(RG_EINVAL, "rg_phase_times: NULL policy");
  if (!pol->phase_valid) return fail(RG_EINVAL, "rg_phase_times: no completed rollout_group call");
  float a = 0.f, b = 0.f;
  HIPTRY(hipEventElapsedTime(&a, pol->phase_ev[0], pol->phase_ev[1]));
  HIPTRY(hipEventElapsedTime(&b, pol->phase_ev[1], pol->phase_ev[2]));
  if (prefill_ms) *prefill_ms = a;
  if (decode_ms) *decode_ms = b;
  return RG_OK;
}

int32_t rg_decode_attention_chunks(int32_t rows, int32_t n_kv, int32_t ctx_max) {
  if (rows < 1 || n_kv < 1 || ctx_max < 1) return fail(RG_EINVAL, "rg_decode_attention_chunks: bad argument");
  return att_row_chunks(row_bucket(rows), n_kv, ctx_max);
}

int rg_kernel_times(const rg_policy* pol, int32_t phase, int32_t kind, double* total_ms, int64_t* launches) {
  if (!pol || phase < 0 || phase >= RG_PROF_PHASES || kind < 0 || kind >= RG_K_COUNT)
    return fail(RG_EINVAL, "rg_kernel_times: bad argument");
  if (total_ms) *total_ms = pol->kt_ms[phase][kind];
  if (launches) *launches = pol->kt_n[phase][kind];
  return RG_OK;
}

}  // extern "C"
