// Paged causal attention over the KV pool, for prefill rows and decode rows
// alike.  Row r attends to positions 0..row_pos[r] through page table
// row_tab[r]; position j lives in page page_tab[tab*tab_stride + j/16], slot
// j % 16, in the key and value slabs of kv_k_off / kv_v_off (16-byte granules
// of 8 dims of a token, resp. 8 tokens of a dim).  Every work item keeps a running softmax
// (max, sum) and an unnormalised output per query head of its GQA group in a
// partial slot of the row; the merge kernel combines a row's slots.
//
// Decode rows split their context in two.  The prompt's full pages (positions
// 0..row_beg[r]-1, shared by all siblings of the prompt) go through the
// prefix kernel: one workgroup per (prompt, kv head, prefix chunk) stages
// each 32-token block of K and V^T once in LDS and scores it against the
// query rows of every active sibling (siblings x GQA heads rows, 16 per
// wave).  The rest (row_beg[r]..row_pos[r]: the copied partial page and the
// sequence's own tokens) goes through the per-row kernel.
//
// bf16 KV: one wave per work item on MFMA 16x16x32.  Scores are formed
// transposed, S^T = K Q^T (tokens x query heads), so each lane ends up holding
// the probabilities of one query head for 8 tokens -- exactly a B fragment of
// O^T = V^T P^T.  The K rows of each 16-token tile are permuted so that lane
// group g ends up with the 8 consecutive tokens 8g..8g+7 of a 32-token block,
// whose V^T fragment is one 16-byte load.  q and p are fp32 values split into
// hi/lo bf16 pairs, so both products keep fp32-level accuracy.  The chunk's
// page ids are read once into LDS and the next block's K and V are loaded
// while the current block is multiplied.
// fp32 KV (fp32 models): a plain per-token VALU kernel.
#include <algorithm>
#include <cstdlib>

#include "rg_device.h"
#include "rg_kernels.h"
#include <hip/hip_ext.h>

namespace {

// Context chunk of a row: its context is cut into at most n_chunks chunks of
// equal length, rounded up to 32 tokens (so chunks start on 32-token blocks)
// and at least 128 tokens; the attention kernel and the merge both use this.
__device__ __forceinline__ int att_chunk_len(int ctx, int n_chunks) {
  return max(128, ((ctx + n_chunks - 1) / n_chunks + 31) & ~31);
}

constexpr int ATT_TILE = 256;   // tokens scored per tile (one per thread)
constexpr int ATT_MAX_REP = 8;  // query heads per kv head
constexpr int ATT_MAX_HD = 256;

template <typename KV>
__device__ __forceinline__ void load8_f32(const KV* p, float* o);
template <> __device__ __forceinline__ void load8_f32<float>(const float* p, float* o) {
  float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w; o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}
template <> __device__ __forceinline__ void load8_f32<bf16_t>(const bf16_t* p, float* o) {
  uint4 u = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = __uint_as_float(w[i] << 16);
    o[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

template <typename KV>
__global__ __launch_bounds__(256) void k_attention(const float* __restrict__ q, int n_q, int n_kv, int hd,
                                                   const KV* __restrict__ pool, KvGeom g, int layer,
                                                   const int32_t* __restrict__ page_tab, int tab_stride,
                                                   const int32_t* __restrict__ row_tab,
                                                   const int32_t* __restrict__ row_pos,
                                                   const int32_t* __restrict__ row_beg, AttPlan plan,
                                                   float* __restrict__ part_o, float* __restrict__ part_ml,
                                                   const int* __restrict__ d_rows) {
  const int r = blockIdx.z;
  // the row's entries (r < the launch's row bound: inside the row arrays)
  // are read alongside the row count and used only once r is below it
  const int rows_now = *d_rows;
  const int pos_r = row_pos[r], beg_r = row_beg[r], tab_r = row_tab[r];
  if ((r >= rows_now) | ((pos_r | beg_r | tab_r) < 0)) return;   // entries of live rows are >= 0
  const int kvh = blockIdx.y, chunk = blockIdx.x;
  const int ctx = pos_r + 1, beg = beg_r;
  const int clen = att_chunk_len(ctx - beg, plan.n_chunks);
  const int c0 = beg + chunk * clen;
  if (c0 >= ctx) return;
  const int c1 = min(ctx, c0 + clen);
  const int rep = n_q / n_kv;
  const int tid = threadIdx.x;
  const float scale = 1.0f / sqrtf((float)hd);

  __shared__ float sq[ATT_MAX_REP * ATT_MAX_HD];
  __shared__ float sp[ATT_MAX_REP * ATT_TILE];
  __shared__ float red[16];
  __shared__ float s_m[ATT_MAX_REP], s_alpha[ATT_MAX_REP], s_l[ATT_MAX_REP];

  for (int i = tid; i < rep * hd; i += blockDim.x)
    sq[i] = q[((int64_t)r * n_q + kvh * rep) * hd + i];
  if (tid < rep) { s_m[tid] = -INFINITY; s_l[tid] = 0.f; }
  const int32_t* tab = page_tab + (int64_t)tab_r * tab_stride;
  const int64_t koff = (int64_t)layer * g.layer_stride + (int64_t)kvh * 16 * hd;
  const int64_t voff = (int64_t)layer * g.layer_stride + ((int64_t)n_kv + kvh) * 16 * hd;

  // each thread owns output slots (h, d) = idx / hd, idx % hd for idx = tid + 256*k
  const int n_own = (rep * hd + 255) / 256;
  float acc[ATT_MAX_REP];
#pragma unroll
  for (int k = 0; k < ATT_MAX_REP; ++k) acc[k] = 0.f;
  __syncthreads();

  for (int t0 = c0; t0 < c1; t0 += ATT_TILE) {
    const int nt = min(ATT_TILE, c1 - t0);
    // ---- scores: one token per thread
    if (tid < nt) {
      const int j = t0 + tid;
      const KV* kp = pool + (int64_t)tab[j >> 4] * g.page_stride + koff;
      float dot[ATT_MAX_REP];
#pragma unroll
      for (int h = 0; h < ATT_MAX_REP; ++h) dot[h] = 0.f;
      for (int d = 0; d < hd; d += 8) {
        float kv8[8];
        load8_f32<KV>(kp + kv_k_off(j & 15, d), kv8);   // dims d .. d+7 of token j
#pragma unroll
        for (int h = 0; h < ATT_MAX_REP; ++h) {
          if (h < rep) {
#pragma unroll
            for (int e = 0; e < 8; ++e) dot[h] = fmaf(sq[h * hd + d + e], kv8[e], dot[h]);
          }
        }
      }
#pragma unroll
      for (int h = 0; h < ATT_MAX_REP; ++h)
        if (h < rep) sp[h * ATT_TILE + tid] = dot[h] * scale;
    }
    __syncthreads();
    // ---- running softmax per head
    for (int h = 0; h < rep; ++h) {
      float v = tid < nt ? sp[h * ATT_TILE + tid] : -INFINITY;
      float mt = block_max(v, red);
      float mnew = fmaxf(s_m[h], mt);
      float p = tid < nt ? expf(v - mnew) : 0.f;
      if (tid < nt) sp[h * ATT_TILE + tid] = p;
      float ps = block_sum(p, red);
      if (tid == 0) {
        float alpha = expf(s_m[h] - mnew);   // 0 on the first tile (exp(-inf))
        s_alpha[h] = alpha;
        s_l[h] = s_l[h] * alpha + ps;
        s_m[h] = mnew;
      }
    }
    __syncthreads();
    // ---- accumulate p * V
    for (int k = 0; k < n_own; ++k) {
      const int idx = tid + 256 * k;
      if (idx < rep * hd) {
        const int h = idx / hd, d = idx % hd;
        float a = acc[k] * s_alpha[h];
        for (int jj = 0; jj < nt; ++jj) {
          const int j = t0 + jj;
          const KV* vp = pool + (int64_t)tab[j >> 4] * g.page_stride + voff;
          a = fmaf(sp[h * ATT_TILE + jj], ld_f32<KV>(vp + kv_v_off(j & 15, d, hd)), a);
        }
        acc[k] = a;
      }
    }
    __syncthreads();
  }
  // ---- write partials
  const int64_t base = ((int64_t)r * plan.n_slots + plan.pre_slots + chunk) * n_q + kvh * rep;
  for (int k = 0; k < n_own; ++k) {
    const int idx = tid + 256 * k;
    if (idx < rep * hd) part_o[base * hd + idx] = acc[k];
  }
  if (tid < rep) {
    part_ml[(base + tid) * 2] = s_m[tid];
    part_ml[(base + tid) * 2 + 1] = s_l[tid];
  }
}


// ---------------------------------------------------------------- MFMA path
// Eight fp32 values as hi = bf16(v) and lo = bf16(v - hi) fragments
// (v_cvt_pk_bf16_f32 rounds to nearest even; v - hi is exact in fp32).
__device__ __forceinline__ void split8(const float* v, bf16x8_t& hi, bf16x8_t& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    l[i] = pack_bf16x2(v[2 * i] - __uint_as_float(h[i] << 16), v[2 * i + 1] - __uint_as_float(h[i] & 0xFFFF0000u));
  }
  hi = __builtin_bit_cast(bf16x8_t, uint4{h[0], h[1], h[2], h[3]});
  lo = __builtin_bit_cast(bf16x8_t, uint4{l[0], l[1], l[2], l[3]});
}

constexpr int ATT_MAX_CHUNK_PAGES = 1024;   // a chunk spans at most 16384 tokens
constexpr int ATT_MAX_MERGE = 1024;         // chunks per row

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Scores are kept in log2 units (q is pre-scaled by log2(e) / sqrt(hd)), so
// probabilities are exp2(s - m).  The running max m may lag the true max by up
// to ATT_SLACK (probabilities then reach 2^ATT_SLACK, far from fp32 overflow):
// the accumulators are rescaled only when a score exceeds m + ATT_SLACK,
// which after the first blocks of a row is rare.  Softmax does not depend on
// the constant subtracted, so only rounding changes.
constexpr float ATT_SLACK = 8.f;
constexpr float ATT_LN2 = 0.693147180559945309f;
constexpr float ATT_LOG2E = 1.44269504088896341f;

// Online-softmax state of one wave: column `col` of the lane is one query
// row; O^T rows 4*grp .. +3 of every 16-dim tile dt.
template <int HD>
struct AttState {
  float m, l;
  f32x4_t o[HD / 16];
};

// Scores S^T of one 32-token block for the lane's query column: s[tt][j] is
// token 8*grp + 4*tt + j of the block.  K fragments kf(tt, kb) supply row
// col of tile tt, dims kb*32 + 8*grp .. +7.
template <int HD, typename KFrag>
__device__ __forceinline__ void att_scores(f32x4_t (&s)[2], const bf16x8_t (&qh)[HD / 32],
                                           const bf16x8_t (&ql)[HD / 32], KFrag kf) {
  f32x4_t a0 = f32x4_t{0.f, 0.f, 0.f, 0.f}, a1 = a0;
#pragma unroll
  for (int kb = 0; kb < HD / 32; ++kb) {   // two independent accumulation chains
    const bf16x8_t k0 = kf(0, kb), k1 = kf(1, kb);
    a0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qh[kb], a0, 0, 0, 0);
    a1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qh[kb], a1, 0, 0, 0);
    a0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, ql[kb], a0, 0, 0, 0);
    a1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, ql[kb], a1, 0, 0, 0);
  }
  s[0] = a0;
  s[1] = a1;
}

// Softmax update and O^T += V^T P^T for one block.  nval = valid tokens among
// the lane group's 8 (only the last block of a range has fewer: `tail`).
// V fragments vf(dt) hold dims dt*16 + col, the lane group's 8 tokens.
template <int HD, typename VFrag>
__device__ __forceinline__ void att_update(AttState<HD>& st, f32x4_t (&s)[2], bool tail, int nval, VFrag vf) {
  if (tail) {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (4 * tt + j >= nval) s[tt][j] = -INFINITY;
  }
  float mloc = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                     fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
  mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
  mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
  if (__any(mloc > st.m + ATT_SLACK)) {
    const float m_new = fmaxf(st.m, mloc);
    const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);   // 0 on the first block (m = -inf)
    st.l *= alpha;
#pragma unroll
    for (int i = 0; i < HD / 16; ++i) st.o[i] *= alpha;
    st.m = m_new;
  }
  float p[8];
  float psum = 0.f;
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float e = __builtin_amdgcn_exp2f(s[tt][j] - st.m);   // exp2(-inf) = 0 for masked tokens
      p[tt * 4 + j] = e;
      psum += e;
    }
  psum += __shfl_xor(psum, 16, 64);
  psum += __shfl_xor(psum, 32, 64);
  st.l += psum;
  bf16x8_t ph, pl;
  split8(p, ph, pl);
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) {
    u32x4_t vv = vf(dt);
    if (tail) {   // zero the slots of masked tokens (their memory may hold anything)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int n2 = nval - 2 * e;   // valid tokens in this dword
        vv[e] = n2 >= 2 ? vv[e] : (n2 == 1 ? (vv[e] & 0xFFFFu) : 0u);
      }
    }
    const bf16x8_t v8 = __builtin_bit_cast(bf16x8_t, vv);
    st.o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v8, ph, st.o[dt], 0, 0, 0);
    st.o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v8, pl, st.o[dt], 0, 0, 0);
  }
}

// Q^T fragments of one query row (a lane's column): dims kb*32 + 8*grp .. +7,
// scaled by log2(e) / sqrt(HD) and split into hi/lo planes.  valid = false
// gives zeros (padding columns; qr must still point at a readable row).
template <int HD>
__device__ __forceinline__ void att_load_q(const float* __restrict__ qr, bool valid, int grp,
                                           bf16x8_t (&qh)[HD / 32], bf16x8_t (&ql)[HD / 32]) {
  const float scale = valid ? ATT_LOG2E / sqrtf((float)HD) : 0.f;
  f32x4_t x[HD / 32][2];   // every load issued before the first conversion
#pragma unroll
  for (int kb = 0; kb < HD / 32; ++kb) {
    x[kb][0] = *reinterpret_cast<const f32x4_t*>(qr + kb * 32 + 8 * grp);
    x[kb][1] = *reinterpret_cast<const f32x4_t*>(qr + kb * 32 + 8 * grp + 4);
  }
#pragma unroll
  for (int kb = 0; kb < HD / 32; ++kb) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) { v[i] = x[kb][0][i] * scale; v[4 + i] = x[kb][1][i] * scale; }
    split8(v, qh[kb], ql[kb]);
  }
}

// The partial of one (row, head, slot): O unnormalised, (m, l) with m in
// natural-log units as the merge expects.
template <int HD>
__device__ __forceinline__ void att_store(const AttState<HD>& st, int64_t base, int grp, float* __restrict__ part_o,
                                          float* __restrict__ part_ml) {
  float* po = part_o + base * HD + 4 * grp;
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) *reinterpret_cast<f32x4_t*>(po + dt * 16) = st.o[dt];
  if (grp == 0) {
    part_ml[base * 2] = st.m * ATT_LN2;
    part_ml[base * 2 + 1] = st.l;
  }
}

// Registers of one 32-token block: K fragments of both 16-token tiles and the
// V^T fragments of every 16-dim output tile.
template <int HD>
struct AttBlock {
  u32x4_t k[2][HD / 32];
  u32x4_t v[HD / 16];
};

// K: A-fragment row i of tile tt is token t0 + 8*(i/4) + 4*tt + (i%4), so that
// the S^T layout leaves lane group grp holding tokens t0+8*grp .. +7; the
// lane's two rows share one page, and lanes 4q..4q+3 read 4 neighbouring
// tokens (64 contiguous bytes of a key slab).  V^T: dims dt*16 + col, tokens
// t0+8*grp .. +7 (one granule).  Tokens past c1 read token c0 instead
// (masked).  t0 is a multiple of 16.
template <int HD>
__device__ __forceinline__ void att_load(AttBlock<HD>& b, const bf16_t* __restrict__ pool, const KvGeom& g,
                                         int64_t koff, int64_t voff, const int* spg, int c0, int c1, int t0,
                                         int col, int grp) {
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    int tok = t0 + 8 * (col >> 2) + 4 * tt + (col & 3);
    if (tok >= c1) tok = c0;
    const bf16_t* kp = pool + (int64_t)spg[(tok - c0) >> 4] * g.page_stride + koff + kv_k_off(tok & 15, 8 * grp);
#pragma unroll
    for (int kb = 0; kb < HD / 32; ++kb) b.k[tt][kb] = *reinterpret_cast<const u32x4_t*>(kp + kb * 4 * 128);
  }
  const int tv = t0 + 8 * grp;
  const int pg = spg[((tv < c1 ? tv : c0) - c0) >> 4];
  const bf16_t* vp = pool + (int64_t)pg * g.page_stride + voff + kv_v_off(tv & 15, col, HD);
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) b.v[dt] = *reinterpret_cast<const u32x4_t*>(vp + dt * 16 * 8);
}

// W > 1: one workgroup of W waves per (row, kv head), wave c taking context
// chunk c of the row's W chunks; at the end the waves merge their (max, sum,
// output) states through LDS in chunk order and write the normalised
// activation, so no merge kernel runs.
// The arguments that locate a work item's row come first (14 dwords, which
// the build preloads into scalar registers at dispatch): the row count and
// the row's entries are then read without a load of the arguments first.
template <int HD, int NB, int W>
__global__ __launch_bounds__(64 * W, NB > 2 ? 1 : 2) void k_attention_mfma(
    const int* __restrict__ d_rows, const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_beg,
    const int32_t* __restrict__ row_tab, int n_chunks, int n_kv, int rows_ub, int n_q, int per_xcd,
    const float* __restrict__ q, const int32_t* __restrict__ page_tab, int tab_stride, const bf16_t* __restrict__ pool,
    KvGeom g, int layer, AttPlan plan, float* __restrict__ part_o, float* __restrict__ part_ml, ActOut out) {
  static_assert(HD % 32 == 0 && HD <= 256, "head_dim");
  // XCD-aware order: the 1-D grid has 8 * per_xcd blocks and blocks are
  // dealt to the 8 XCDs round-robin, so XCD x = b % 8 takes the contiguous
  // work range [x*per_xcd, (x+1)*per_xcd): neighbouring rows (siblings of one
  // prompt) share an XCD, whose L2 then holds their shared prefix.  The
  // launch keeps every index below 2^31.
  const int b = (int)blockIdx.x;
  const int w = (b % 8) * per_xcd + b / 8;
  const int wave = W == 1 ? 0 : (int)(threadIdx.x >> 6);
  int chunk, kvh, r;
  if constexpr (W == 1) {
    if (w >= n_chunks * n_kv * rows_ub) return;
    chunk = w % n_chunks;
    kvh = (w / n_chunks) % n_kv;
    r = w / (n_chunks * n_kv);
  } else {   // the workgroup's (row, kv head); n_chunks == W
    if (w >= n_kv * rows_ub) return;
    chunk = wave;
    kvh = w % n_kv;
    r = w / n_kv;
  }
  // The row's entries (r < rows_ub: inside the row arrays) are read
  // alongside the row count and used only once r is below it.  Rows below
  // the count hold entries >= 0, so the sign test only joins their loads to
  // the row test's one wait (the compiler would otherwise sink them past it).
  const int rows_now = *d_rows;
  const int pos_r = row_pos[r], beg_r = row_beg[r], tab_r = row_tab[r];
  if ((r >= rows_now) | ((pos_r | beg_r | tab_r) < 0)) return;   // uniform over the workgroup
  const int ctx = pos_r + 1, beg = beg_r;
  const int clen = att_chunk_len(ctx - beg, n_chunks);
  const int c0 = beg + chunk * clen;                // a multiple of 16
  if constexpr (W == 1)
    if (c0 >= ctx) return;
  const bool live = c0 < ctx;                       // W > 1: an empty chunk still joins the merge
  const int c1 = live ? min(ctx, c0 + clen) : c0;
  const int rep = n_q / n_kv;
  const int lane = threadIdx.x & 63, col = lane & 15, grp = lane >> 4;

  // page ids of the chunk, once (each wave its own)
  __shared__ int spg_w[W][ATT_MAX_CHUNK_PAGES];
  int* spg = spg_w[wave];
  {
    const int32_t* tab = page_tab + (int64_t)tab_r * tab_stride + (c0 >> 4);
    const int npg = (c1 - c0 + 15) >> 4;
    for (int i = lane; i < npg; i += 64) spg[i] = tab[i];
    __syncthreads();
  }
  const int64_t koff = (int64_t)layer * g.layer_stride + (int64_t)kvh * 16 * HD;
  const int64_t voff = (int64_t)layer * g.layer_stride + ((int64_t)n_kv + kvh) * 16 * HD;
  // NB register blocks in a ring: the next NB-1 blocks' loads are in flight
  // while one block is multiplied out (a launch holds about one wave per
  // SIMD, so latency is hidden inside the wave)
  AttBlock<HD> bk[NB];
  if (live) att_load<HD>(bk[0], pool, g, koff, voff, spg, c0, c1, c0, col, grp);   // first block in flight during the q set-up
  // Q^T fragments (lanes >= rep: zero padding columns), parked in LDS in lane
  // order so that each lane reads back its own 16-byte pieces
  __shared__ __attribute__((aligned(16))) u32x4_t sq_w[W][2][HD / 32][64];
  auto& sq = sq_w[wave];
  {
    bf16x8_t qh[HD / 32], ql[HD / 32];
    att_load_q<HD>(q + ((int64_t)r * n_q + kvh * rep + min(col, rep - 1)) * HD, col < rep, grp, qh, ql);
#pragma unroll
    for (int kb = 0; kb < HD / 32; ++kb) {
      sq[0][kb][lane] = __builtin_bit_cast(u32x4_t, qh[kb]);
      sq[1][kb][lane] = __builtin_bit_cast(u32x4_t, ql[kb]);
    }
  }

  AttState<HD> st;
  st.m = -INFINITY;
  st.l = 0.f;
#pragma unroll
  for (int i = 0; i < HD / 16; ++i) st.o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // two register blocks in turn: the next block's loads are in flight while
  // the current one is multiplied out
  auto step = [&](const AttBlock<HD>& blk, int t0) {
    f32x4_t s[2];
    bf16x8_t qh[HD / 32], ql[HD / 32];
    asm volatile("" ::: "memory");   // re-read q from LDS each block rather than pinning it in registers
#pragma unroll
    for (int kb = 0; kb < HD / 32; ++kb) {
      qh[kb] = __builtin_bit_cast(bf16x8_t, sq[0][kb][lane]);
      ql[kb] = __builtin_bit_cast(bf16x8_t, sq[1][kb][lane]);
    }
    att_scores<HD>(s, qh, ql, [&](int tt, int kb) { return __builtin_bit_cast(bf16x8_t, blk.k[tt][kb]); });
    att_update<HD>(st, s, t0 + 32 > c1, min(8, max(0, c1 - (t0 + 8 * grp))), [&](int dt) { return blk.v[dt]; });
  };
#pragma unroll
  for (int j = 1; j < NB - 1; ++j)
    if (c0 + 32 * j < c1) att_load<HD>(bk[j], pool, g, koff, voff, spg, c0, c1, c0 + 32 * j, col, grp);
  for (int t0 = c0; t0 < c1; t0 += 32 * NB) {
    bool done = false;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int tb = t0 + 32 * j;
      if (!done && tb < c1) {
        const int tn = tb + 32 * (NB - 1);
        if (tn < c1) att_load<HD>(bk[(j + NB - 1) % NB], pool, g, koff, voff, spg, c0, c1, tn, col, grp);
        step(bk[j], tb);
      } else {
        done = true;
      }
    }
    if (done) break;
  }
  if constexpr (W > 1) {
    // Merge of the W chunk states, in chunk order.  Each wave parks its state
    // in its own q area (free after its last block): output rows [col][HD]
    // for its query heads, then (m, l) per head, m in log2 units.
    float* so = reinterpret_cast<float*>(&sq[0][0][0]);
    float* sml = so + ATT_MAX_REP * HD;
    static_assert(ATT_MAX_REP * HD * 4 + ATT_MAX_REP * 8 <= 2 * (HD / 32) * 64 * 16, "state fits the q area");
    if (col < rep) {
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
        for (int e = 0; e < 4; ++e) so[col * HD + dt * 16 + 4 * grp + e] = st.o[dt][e];
      if (grp == 0) {
        sml[2 * col] = st.m;
        sml[2 * col + 1] = st.l;
      }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < rep * HD; i += 64 * W) {
      const int h = i / HD, d = i - h * HD;
      float M = -INFINITY;
#pragma unroll
      for (int c = 0; c < W; ++c)
        M = fmaxf(M, reinterpret_cast<const float*>(&sq_w[c][0][0][0])[ATT_MAX_REP * HD + 2 * h]);
      float L = 0.f, o = 0.f;
#pragma unroll
      for (int c = 0; c < W; ++c) {
        const float* sc = reinterpret_cast<const float*>(&sq_w[c][0][0][0]);
        const float mc = sc[ATT_MAX_REP * HD + 2 * h];
        const float f = mc == -INFINITY ? 0.f : exp2f(mc - M);   // an empty chunk weighs 0
        L += f * sc[ATT_MAX_REP * HD + 2 * h + 1];
        o += f * sc[h * HD + d];
      }
      act_store<1>(out, ((int64_t)r * n_q + kvh * rep + h) * HD + d, o / L);
    }
    return;
  }
  if (col < rep) {
    if (plan.n_slots == 1) {   // the whole context in one work item: normalise and write the activation
      const float inv = 1.0f / st.l;
      bf16_t* o = (bf16_t*)out.base + ((int64_t)r * n_q + kvh * rep + col) * HD + 4 * grp;
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) {
        uint32_t h[2], l[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const float v0 = st.o[dt][2 * e] * inv, v1 = st.o[dt][2 * e + 1] * inv;
          h[e] = pack_bf16x2(v0, v1);
          l[e] = pack_bf16x2(v0 - __uint_as_float(h[e] << 16), v1 - __uint_as_float(h[e] & 0xFFFF0000u));
        }
        *reinterpret_cast<uint2*>(o + dt * 16) = uint2{h[0], h[1]};
        *reinterpret_cast<uint2*>(o + out.plane + dt * 16) = uint2{l[0], l[1]};
      }
    } else {
      att_store<HD>(st, ((int64_t)r * plan.n_slots + plan.pre_slots + chunk) * n_q + kvh * rep + col, grp, part_o,
                    part_ml);
    }
  }
}


// Staging of one 32-token block of K and V^T through LDS, shared by the
// prefix and row-tile passes.  The block is 8*HD 16-byte pieces: 4*HD of K
// (LDS row L = the S^T fragment lane order of its token, 8 dims each) then
// 4*HD of V^T (dim dd, 8 tokens each); thread tid takes pieces tid + k*nthr.
// Blocks start on 32-token boundaries of a range that starts on a page, so a
// piece's page within the block (0 or 1), its offset inside the page and its
// LDS slot are the same for every block: they are worked out once
// (KvStagePlan), and a block's fetch is one page-id read and one address add
// per piece.  Consecutive threads fill consecutive K rows, which keeps the
// LDS writes free of bank conflicts.  Page ids past the range repeat its
// last page (KV_STAGE_PAD), so a tail block needs no clamp: its extra tokens
// are masked by the caller.
template <int HD>
struct KvStage {
  static constexpr int KROW = HD + 8;           // LDS row stride of K (elements)
  static constexpr int VROW = 40;               // LDS row stride of V^T (32 tokens + 8)
  static constexpr int VBASE = 32 * KROW;       // V^T rows follow the K rows in a block buffer
  static constexpr int BUF = VBASE + HD * VROW; // elements per block buffer
  static constexpr int PIECES = 8 * HD;
  static constexpr int MAXP = PIECES / 256;     // pieces per thread (at least 4 waves)
};

// Page ids of [c0, c1) (c0 a multiple of 32 from the table start `tab`),
// padded to whole 32-token blocks with the last page.
__device__ __forceinline__ void kv_stage_pages(int* spg, const int32_t* __restrict__ tab, int c0, int c1, int tid,
                                               int nthr) {
  const int npg = (c1 - c0 + 15) >> 4;
  const int npad = ((c1 - c0 + 31) >> 5) << 1;
  for (int i = tid; i < npad; i += nthr) spg[i] = tab[min(i, npg - 1)];
}

template <int HD>
struct KvStagePlan {
  int64_t off[KvStage<HD>::MAXP];   // element offset of the piece inside its page
  int pg[KvStage<HD>::MAXP];        // page of the piece within the block: 0 or 1
  int dst[KvStage<HD>::MAXP];       // LDS element offset inside a block buffer
  bool on[KvStage<HD>::MAXP];       // the piece exists
};

template <int HD>
__device__ __forceinline__ void kv_stage_plan(KvStagePlan<HD>& pl, int64_t koff, int64_t voff, int tid, int nthr) {
#pragma unroll
  for (int k = 0; k < KvStage<HD>::MAXP; ++k) {
    int pc = tid + k * nthr;
    pl.on[k] = pc < KvStage<HD>::PIECES;
    pc = pl.on[k] ? pc : 0;                      // spare slots load piece 0 (never stored)
    if (pc < 4 * HD) {
      const int L = pc & 31, ck = pc >> 5;
      const int tk = (((L & 15) >> 2) << 3) | ((L >> 4) << 2) | (L & 3);   // the token whose fragment row is L
      pl.pg[k] = tk >> 4;
      pl.off[k] = koff + kv_k_off(tk & 15, ck * 8);
      pl.dst[k] = L * KvStage<HD>::KROW + ck * 8;
    } else {
      const int pv = pc - 4 * HD, dd = pv % HD, q4 = pv / HD;
      pl.pg[k] = q4 >> 1;
      pl.off[k] = voff + kv_v_off((q4 * 8) & 15, dd, HD);
      pl.dst[k] = KvStage<HD>::VBASE + dd * KvStage<HD>::VROW + q4 * 8;
    }
  }
}

// Pieces of the block starting at token t0 (spg indexes pages from c0).
template <int HD>
__device__ __forceinline__ void kv_stage_fetch(u32x4_t (&rg)[KvStage<HD>::MAXP], const KvStagePlan<HD>& pl,
                                               const bf16_t* __restrict__ pool, int64_t page_stride, const int* spg,
                                               int c0, int t0) {
  const int* sp = spg + ((t0 - c0) >> 4);
#pragma unroll
  for (int k = 0; k < KvStage<HD>::MAXP; ++k)
    rg[k] = *reinterpret_cast<const u32x4_t*>(pool + (int64_t)sp[pl.pg[k]] * page_stride + pl.off[k]);
}

template <int HD>
__device__ __forceinline__ void kv_stage_stash(const u32x4_t (&rg)[KvStage<HD>::MAXP], const KvStagePlan<HD>& pl,
                                               bf16_t* buf) {
#pragma unroll
  for (int k = 0; k < KvStage<HD>::MAXP; ++k)
    if (pl.on[k]) *reinterpret_cast<u32x4_t*>(buf + pl.dst[k]) = rg[k];
}

// Prefix pass.  Workgroup (chunk, kv head, prompt p, row block b) with W
// waves; wave w scores query rows 16(bW + w) .. +15 of the group (row i =
// sibling i / rep, GQA head i % rep).
// Per 32-token block every thread stages a few 16-byte pieces of K (LDS row
// = the fragment lane order of S^T, so one quarter-wave reads 16 consecutive
// rows) and V^T (padded rows) for the next block in registers while the
// waves multiply the current block out of LDS (two LDS buffers).
constexpr int ATT_PRE_MAX_WAVES = 8;

template <int HD>
__global__ __launch_bounds__(64 * ATT_PRE_MAX_WAVES) void k_attention_prefix(const float* __restrict__ q, int n_q, int n_kv,
                                                         const bf16_t* __restrict__ pool, KvGeom g, int layer,
                                                         const int32_t* __restrict__ page_tab, int tab_stride,
                                                         int tab_base, const int32_t* __restrict__ plen,
                                                         const int32_t* __restrict__ grp_row0,
                                                         const int32_t* __restrict__ grp_row1, int n_rblk,
                                                         AttPlan plan, float* __restrict__ part_o,
                                                         float* __restrict__ part_ml) {
  constexpr int KROW = KvStage<HD>::KROW, VROW = KvStage<HD>::VROW;
  __shared__ __attribute__((aligned(16))) bf16_t sKV[2][KvStage<HD>::BUF];
  __shared__ int spg[64];

  const int c = blockIdx.x, kvh = blockIdx.y, p = blockIdx.z / n_rblk, rb = blockIdx.z % n_rblk;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nthr = blockDim.x;
  const int r0 = grp_row0[p], r1 = grp_row1[p];
  const int rep = n_q / n_kv;
  const int q0 = rb * (nthr / 4);                // first query row of this block (16 per wave)
  const int nrows = (r1 - r0) * rep;
  if (q0 >= nrows) return;
  const int pref = (plen[p] >> 4) << 4;
  const int c0 = c * plan.pre_chunk;
  if (c0 >= pref) return;
  const int c1 = min(pref, c0 + plan.pre_chunk);
  const int col = lane & 15, grp = lane >> 4;
  const bool active = q0 + wave * 16 < nrows;
  const int qi = q0 + wave * 16 + col;
  const bool qv = qi < nrows;
  const int row = r0 + (qv ? qi / rep : 0), head = kvh * rep + (qv ? qi % rep : 0);

  kv_stage_pages(spg, page_tab + (int64_t)(tab_base + p) * tab_stride + (c0 >> 4), c0, c1, tid, nthr);
  bf16x8_t qh[HD / 32], ql[HD / 32];
  att_load_q<HD>(q + ((int64_t)row * n_q + head) * HD, qv, grp, qh, ql);
  __syncthreads();   // page ids
  const int64_t koff = (int64_t)layer * g.layer_stride + (int64_t)kvh * 16 * HD;
  const int64_t voff = (int64_t)layer * g.layer_stride + ((int64_t)n_kv + kvh) * 16 * HD;

  KvStagePlan<HD> pl;
  kv_stage_plan<HD>(pl, koff, voff, tid, nthr);
  u32x4_t rg[KvStage<HD>::MAXP];
  auto fetch = [&](int t0) { kv_stage_fetch<HD>(rg, pl, pool, g.page_stride, spg, c0, t0); };
  auto stash = [&](int buf) { kv_stage_stash<HD>(rg, pl, sKV[buf]); };

  AttState<HD> st;
  st.m = -INFINITY;
  st.l = 0.f;
#pragma unroll
  for (int i = 0; i < HD / 16; ++i) st.o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  fetch(c0);
  int buf = 0;
  for (int t0 = c0; t0 < c1; t0 += 32, buf ^= 1) {
    stash(buf);
    __syncthreads();                             // block t0 in LDS; the other buffer is free
    if (t0 + 32 < c1) fetch(t0 + 32);
    if (!active) continue;
    f32x4_t s[2];
    const bf16_t* kb0 = &sKV[buf][col * KROW + 8 * grp];
    att_scores<HD>(s, qh, ql, [&](int tt, int kb) {
      return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4_t*>(kb0 + 16 * tt * KROW + kb * 32));
    });
    const bf16_t* vb0 = &sKV[buf][KvStage<HD>::VBASE + col * VROW + 8 * grp];
    att_update<HD>(st, s, t0 + 32 > c1, min(8, max(0, c1 - (t0 + 8 * grp))),
                   [&](int dt) { return *reinterpret_cast<const u32x4_t*>(vb0 + dt * 16 * VROW); });
  }
  if (active && qv) att_store<HD>(st, ((int64_t)row * plan.n_slots + c) * n_q + head, grp, part_o, part_ml);
}

// Row tiles of one sequence (prefill-style rows: many consecutive positions
// of a sequence in one launch).  Workgroup (tile, kv head): the tile's rows
// tile_r0[k] .. +tile_nr[k]-1 hold consecutive positions of one page table
// row; its nr x rep query rows (row i = tile row i / rep, GQA head i % rep)
// are scored 16 per wave against each 32-token block of K and V^T, staged
// once in LDS for all waves (double buffered, as in the prefix pass).  Query
// row i sees tokens 0 .. row_pos of its row (causal mask per column).  The
// whole context is one work item, so the normalised output goes straight to
// the activation planes.
constexpr int ATT_TILE_MAX_WAVES = 12;

// Positions per row tile: 32 while the tile's query rows (positions x GQA
// heads) fit ATT_TILE_MAX_WAVES waves of 16, else 16.
int att_tile_rows_for(int rep) { return 32 * rep <= 16 * ATT_TILE_MAX_WAVES ? 32 : 16; }

template <int HD>
__global__ __launch_bounds__(64 * ATT_TILE_MAX_WAVES) void k_attention_tile(
    const float* __restrict__ q, int n_q, int n_kv, const bf16_t* __restrict__ pool, KvGeom g, int layer,
    const int32_t* __restrict__ page_tab, int tab_stride, const int32_t* __restrict__ row_tab,
    const int32_t* __restrict__ row_pos, const int32_t* __restrict__ tile_r0, const int32_t* __restrict__ tile_nr,
    const int* __restrict__ d_tiles, ActOut out) {
  constexpr int KROW = KvStage<HD>::KROW, VROW = KvStage<HD>::VROW;
  __shared__ __attribute__((aligned(16))) bf16_t sKV[2][KvStage<HD>::BUF];
  __shared__ int spg[ATT_MAX_CHUNK_PAGES];

  // XCD-aware order: consecutive tiles (one sequence's rows) share an XCD
  const int64_t b = blockIdx.x;
  const int64_t per_xcd = (int64_t)gridDim.x / 8;
  const int64_t w = (b % 8) * per_xcd + b / 8;
  const int k = (int)(w / n_kv), kvh = (int)(w % n_kv);
  if (k >= *d_tiles) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nthr = blockDim.x;
  const int rep = n_q / n_kv;
  const int r0 = tile_r0[k], nr = tile_nr[k];
  const int nrows = nr * rep;
  const int c1 = row_pos[r0 + nr - 1] + 1;      // the tile's last row sees the longest context
  const int col = lane & 15, grp = lane >> 4;
  const bool active = wave * 16 < nrows;
  const int qi = wave * 16 + col;
  const bool qv = qi < nrows;
  const int row = r0 + (qv ? qi / rep : 0), head = kvh * rep + (qv ? qi % rep : 0);
  const int climit = row_pos[row] + 1;

  kv_stage_pages(spg, page_tab + (int64_t)row_tab[r0] * tab_stride, 0, c1, tid, nthr);
  bf16x8_t qh[HD / 32], ql[HD / 32];
  att_load_q<HD>(q + ((int64_t)row * n_q + head) * HD, qv, grp, qh, ql);
  __syncthreads();   // page ids
  const int64_t koff = (int64_t)layer * g.layer_stride + (int64_t)kvh * 16 * HD;
  const int64_t voff = (int64_t)layer * g.layer_stride + ((int64_t)n_kv + kvh) * 16 * HD;

  KvStagePlan<HD> pl;
  kv_stage_plan<HD>(pl, koff, voff, tid, nthr);
  u32x4_t rg[KvStage<HD>::MAXP];
  auto fetch = [&](int t0) { kv_stage_fetch<HD>(rg, pl, pool, g.page_stride, spg, 0, t0); };
  auto stash = [&](int buf) { kv_stage_stash<HD>(rg, pl, sKV[buf]); };

  AttState<HD> st;
  st.m = -INFINITY;
  st.l = 0.f;
#pragma unroll
  for (int i = 0; i < HD / 16; ++i) st.o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // two register sets in turn keep the next two blocks' loads in flight
  // while one block is multiplied out of LDS
  u32x4_t rg2[KvStage<HD>::MAXP];
  auto fetch2 = [&](int t0) { kv_stage_fetch<HD>(rg2, pl, pool, g.page_stride, spg, 0, t0); };
  auto stash2 = [&](int buf) { kv_stage_stash<HD>(rg2, pl, sKV[buf]); };
  auto block = [&](int buf, int t0) {
    if (!active) return;
    f32x4_t s[2];
    const bf16_t* kb0 = &sKV[buf][col * KROW + 8 * grp];
    att_scores<HD>(s, qh, ql, [&](int tt, int kb) {
      return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4_t*>(kb0 + 16 * tt * KROW + kb * 32));
    });
    if (t0 + 32 > climit) {                      // causal mask of this column (token 0 is always visible)
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (t0 + 8 * grp + 4 * tt + j >= climit) s[tt][j] = -INFINITY;
    }
    const bf16_t* vb0 = &sKV[buf][KvStage<HD>::VBASE + col * VROW + 8 * grp];
    att_update<HD>(st, s, t0 + 32 > c1, min(8, max(0, c1 - (t0 + 8 * grp))),
                   [&](int dt) { return *reinterpret_cast<const u32x4_t*>(vb0 + dt * 16 * VROW); });
  };
  fetch(0);
  if (32 < c1) fetch2(32);
  for (int t0 = 0; t0 < c1; t0 += 64) {
    stash(0);
    __syncthreads();                             // block t0 in buffer 0; buffer 1 is free
    if (t0 + 64 < c1) fetch(t0 + 64);
    block(0, t0);
    if (t0 + 32 >= c1) break;
    stash2(1);
    __syncthreads();                             // block t0 + 32 in buffer 1; buffer 0 is free
    if (t0 + 96 < c1) fetch2(t0 + 96);
    block(1, t0 + 32);
  }
  if (active && qv) {
    const float inv = 1.0f / st.l;
    bf16_t* o = (bf16_t*)out.base + ((int64_t)row * n_q + head) * HD + 4 * grp;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      uint32_t h[2], l[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const float v0 = st.o[dt][2 * e] * inv, v1 = st.o[dt][2 * e + 1] * inv;
        h[e] = pack_bf16x2(v0, v1);
        l[e] = pack_bf16x2(v0 - __uint_as_float(h[e] << 16), v1 - __uint_as_float(h[e] & 0xFFFF0000u));
      }
      *reinterpret_cast<uint2*>(o + dt * 16) = uint2{h[0], h[1]};
      *reinterpret_cast<uint2*>(o + out.plane + dt * 16) = uint2{l[0], l[1]};
    }
  }
}

template <int SPLIT>
__global__ void k_attn_merge(const int* __restrict__ d_rows, const int32_t* __restrict__ row_pos,
                             const int32_t* __restrict__ row_beg, const float* __restrict__ part_o,
                             const float* __restrict__ part_ml, int n_q, int hd, AttPlan plan, ActOut out) {
  const int r = blockIdx.x;
  const int rows_now = *d_rows;
  const int pos_r = row_pos[r], beg_r = row_beg[r];   // r < the row bound: inside the row arrays
  if ((r >= rows_now) | ((pos_r | beg_r) < 0)) return;   // entries of live rows are >= 0
  const int h = blockIdx.y;
  const int ctx = pos_r + 1, beg = beg_r;
  const int clen = att_chunk_len(ctx - beg, plan.n_chunks);
  const int npre = plan.pre_slots ? (beg + plan.pre_chunk - 1) / plan.pre_chunk : 0;   // prefix slots written
  const int nc = npre + (ctx - beg + clen - 1) / clen;                                  // slots holding context
  __shared__ float sw[ATT_MAX_MERGE];       // slot weights exp(m_c - M)
  // slot c of the merge: prefix slot c < npre, else private slot pre_slots + c - npre
  const int gap = plan.pre_slots - npre;
  const int64_t rb = (int64_t)r * plan.n_slots;
#define RG_SLOT(c) ((c) < npre ? (c) : (c) + gap)
  float m = -INFINITY;
  for (int c = threadIdx.x; c < nc; c += blockDim.x) m = fmaxf(m, part_ml[((rb + RG_SLOT(c)) * n_q + h) * 2]);
  __shared__ float red[16];
  const float M = block_max(m, red);
  float l = 0.f;
  for (int c = threadIdx.x; c < nc; c += blockDim.x) {
    const float* ml = part_ml + ((rb + RG_SLOT(c)) * n_q + h) * 2;
    const float w = expf(ml[0] - M);
    sw[c] = w;
    l += w * ml[1];
  }
  const float invL = 1.0f / block_sum(l, red);
  for (int d = threadIdx.x; d < hd; d += blockDim.x) {
    float o0 = 0.f, o1 = 0.f, o2 = 0.f, o3 = 0.f;   // independent sums keep several loads in flight
    int c = 0;
    for (; c + 4 <= nc; c += 4) {
      o0 += sw[c] * part_o[((rb + RG_SLOT(c)) * n_q + h) * hd + d];
      o1 += sw[c + 1] * part_o[((rb + RG_SLOT(c + 1)) * n_q + h) * hd + d];
      o2 += sw[c + 2] * part_o[((rb + RG_SLOT(c + 2)) * n_q + h) * hd + d];
      o3 += sw[c + 3] * part_o[((rb + RG_SLOT(c + 3)) * n_q + h) * hd + d];
    }
    for (; c < nc; ++c) o0 += sw[c] * part_o[((rb + RG_SLOT(c)) * n_q + h) * hd + d];
    act_store<SPLIT>(out, ((int64_t)r * n_q + h) * hd + d, ((o0 + o1) + (o2 + o3)) * invL);
  }
#undef RG_SLOT
}

}  // namespace

// One kernel launch; with armed timing events they time the dispatch itself.
template <typename F, typename... Args>
void att_launch(F kernel, dim3 grid, dim3 block, hipStream_t st, Args... args) {
  hipEvent_t e0, e1;
  if (rg_take_launch_events(&e0, &e1))
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, e0, e1, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
}

hipError_t launch_attention(int dtype, const float* q, int n_q, int n_kv, int head_dim, const void* kv_pool,
                            KvGeom g, int layer, const int32_t* page_tab, int tab_stride,
                            const int32_t* row_tab, const int32_t* row_pos, const int32_t* row_beg, int max_ctx,
                            AttPlan plan, float* part_o, float* part_ml, void* out, int64_t a_plane,
                            const int* d_rows, int rows_ub, hipStream_t st) {
  const int n_chunks = plan.n_chunks;
  if (n_chunks < 1 || plan.n_slots != plan.pre_slots + n_chunks || plan.n_slots > ATT_MAX_MERGE ||
      std::max(128, (max_ctx + n_chunks - 1) / n_chunks + 31) > 16 * ATT_MAX_CHUNK_PAGES)
    return hipErrorInvalidValue;
  if (rows_ub <= 0) return hipSuccess;
  dim3 grid(n_chunks, n_kv, rows_ub);
  if (dtype == 1) {
    // two 16-slot pages per 32-token block
    if (g.page_tok != 16) return hipErrorInvalidValue;
    const int W = att_merges_in_kernel(dtype, plan, rows_ub, n_kv) ? n_chunks : 1;
    const int64_t nb = (int64_t)(W == 1 ? n_chunks : 1) * n_kv * rows_ub;
    if (nb > INT32_MAX - 8) return hipErrorInvalidValue;
    const int per_xcd = (int)((nb + 7) / 8);
    const dim3 grid1((unsigned)(8 * per_xcd));
#define RG_ATT_W(HD, WV)                                                                                          \
    att_launch(k_attention_mfma<HD, 2, WV>, grid1, dim3(64 * WV), st, d_rows, row_pos, row_beg, row_tab, n_chunks, \
               n_kv, rows_ub, n_q, per_xcd, q, page_tab, tab_stride, (const bf16_t*)kv_pool, g, layer, plan, part_o, \
               part_ml, ActOut{out, a_plane})
#define RG_ATT_MFMA(HD)                                                                                          \
    switch (W) {                                                                                                 \
      case 1: RG_ATT_W(HD, 1); break;                                                                            \
      case 2: RG_ATT_W(HD, 2); break;                                                                            \
      case 3: RG_ATT_W(HD, 3); break;                                                                            \
      case 4: RG_ATT_W(HD, 4); break;                                                                            \
      case 5: RG_ATT_W(HD, 5); break;                                                                            \
      case 6: RG_ATT_W(HD, 6); break;                                                                            \
      case 7: RG_ATT_W(HD, 7); break;                                                                            \
      default: RG_ATT_W(HD, 8); break;                                                                           \
    }
    switch (head_dim) {
      case 64: RG_ATT_MFMA(64); break;
      case 128: RG_ATT_MFMA(128); break;
      default: return hipErrorInvalidValue;
    }
#undef RG_ATT_MFMA
#undef RG_ATT_W
  } else
    att_launch(k_attention<float>, grid, dim3(256), st, q, n_q, n_kv, head_dim, (const float*)kv_pool, g, layer,
               page_tab, tab_stride, row_tab, row_pos, row_beg, plan, part_o, part_ml, d_rows);
  return hipGetLastError();
}

hipError_t launch_attention_prefix(const float* q, int n_q, int n_kv, int head_dim, const void* kv_pool, KvGeom g,
                                   int layer, const int32_t* page_tab, int tab_stride, int tab_base,
                                   const int32_t* plen, const int32_t* grp_row0, const int32_t* grp_row1, int P,
                                   int max_group_rows, AttPlan plan, float* part_o, float* part_ml, hipStream_t st) {
  if (plan.pre_slots <= 0) return hipSuccess;
  const int tiles = (max_group_rows * (n_q / n_kv) + 15) / 16;   // 16-row query tiles of the largest group
  if (g.page_tok != 16 || plan.pre_chunk <= 0 || plan.pre_chunk % 32 || plan.pre_chunk > 1024 || tiles < 1 ||
      P < 1)
    return hipErrorInvalidValue;
  const int n_rblk = (tiles + ATT_PRE_MAX_WAVES - 1) / ATT_PRE_MAX_WAVES;
  const int waves = std::max(4, (tiles + n_rblk - 1) / n_rblk);
  if ((int64_t)P * n_rblk > 65535) return hipErrorInvalidValue;
  dim3 grid(plan.pre_slots, n_kv, P * n_rblk);
  const bf16_t* pool = (const bf16_t*)kv_pool;
  switch (head_dim) {
    case 64:
      att_launch(k_attention_prefix<64>, grid, dim3(64 * waves), st, q, n_q, n_kv, pool, g, layer, page_tab,
                 tab_stride, tab_base, plen, grp_row0, grp_row1, n_rblk, plan, part_o, part_ml);
      break;
    case 128:
      att_launch(k_attention_prefix<128>, grid, dim3(64 * waves), st, q, n_q, n_kv, pool, g, layer, page_tab,
                 tab_stride, tab_base, plen, grp_row0, grp_row1, n_rblk, plan, part_o, part_ml);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn_merge(int dtype, const float* part_o, const float* part_ml, int n_q, int head_dim,
                             const int32_t* row_pos, const int32_t* row_beg, AttPlan plan, void* out, int64_t a_plane,
                             const int* d_rows, int rows_ub, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  if (plan.n_chunks < 1 || plan.n_slots > ATT_MAX_MERGE) return hipErrorInvalidValue;
  dim3 grid(rows_ub, n_q);
  int threads = head_dim >= 64 ? 64 * ((head_dim + 63) / 64) : 64;
  const ActOut o{out, a_plane};
  if (dtype == 1)
    hipLaunchKernelGGL(k_attn_merge<1>, grid, dim3(threads), 0, st, d_rows, row_pos, row_beg, part_o, part_ml, n_q,
                       head_dim, plan, o);
  else
    hipLaunchKernelGGL(k_attn_merge<0>, grid, dim3(threads), 0, st, d_rows, row_pos, row_beg, part_o, part_ml, n_q,
                       head_dim, plan, o);
  return hipGetLastError();
}

hipError_t launch_attention_tile(const float* q, int n_q, int n_kv, int head_dim, const void* kv_pool, KvGeom g,
                                 int layer, const int32_t* page_tab, int tab_stride, const int32_t* row_tab,
                                 const int32_t* row_pos, const int32_t* tile_r0, const int32_t* tile_nr,
                                 const int* d_tiles, int tiles_ub, int max_ctx, void* out, int64_t a_plane,
                                 hipStream_t st) {
  if (tiles_ub <= 0) return hipSuccess;
  const int rep = n_q / n_kv;
  const int rows = att_tile_rows_for(rep);
  if (rows * rep > 16 * ATT_TILE_MAX_WAVES || max_ctx > 16 * ATT_MAX_CHUNK_PAGES) return hipErrorInvalidValue;
  const int waves = std::max(4, (rows * rep + 15) / 16);
  const int64_t items = (int64_t)tiles_ub * n_kv;
  const unsigned blocks = (unsigned)((items + 7) / 8 * 8);
  const ActOut o{out, a_plane};
  if (head_dim == 128)
    att_launch(k_attention_tile<128>, dim3(blocks), dim3(64 * waves), st, q, n_q, n_kv, (const bf16_t*)kv_pool, g,
               layer, page_tab, tab_stride, row_tab, row_pos, tile_r0, tile_nr, d_tiles, o);
  else if (head_dim == 64)
    att_launch(k_attention_tile<64>, dim3(blocks), dim3(64 * waves), st, q, n_q, n_kv, (const bf16_t*)kv_pool, g,
               layer, page_tab, tab_stride, row_tab, row_pos, tile_r0, tile_nr, d_tiles, o);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

int att_tile_rows(int n_q, int n_kv) { return att_tile_rows_for(n_q / n_kv); }

// About ATT_ITEMS_TARGET work items (fewer, longer chunks measured faster than
// filling every wave slot: less partial traffic and per-item set-up), at least
// ~256 tokens each for the longest context, at most 16000 tokens each.  From
// 512 to 2048 (row, kv head) pairs, where the chunks of a row are merged
// inside the attention kernel, rows take at least two chunks: twice the waves
// per CU and no merge launch (1.5B at 384-512 rows: 64.5 -> 60.1 us a launch).
int att_row_chunks(int rows_ub, int n_kv, int ctx_max) {
  const int64_t items = (int64_t)rows_ub * n_kv;
  int n = (int)std::min<int64_t>((ATT_ITEMS_TARGET + items / 2) / items, (ctx_max + 255) / 256);
  if (items >= 512 && items <= 2048 && ctx_max >= 512) n = std::max(n, 2);
  return std::max<int>({1, n, (ctx_max + 15999) / 16000});
}
