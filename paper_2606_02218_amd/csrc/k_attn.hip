// Paged causal attention over the KV pool, for prefill rows and decode rows
// alike.  Work item = (row, kv head, chunk of the row's context); it keeps a
// running softmax (max, sum) and an unnormalised output per query head of the
// GQA group, and the merge kernel combines the chunks.  Context positions
// 0..row_pos[r] of page table row_tab[r]; position j lives in page
// page_tab[tab*tab_stride + j/page_tok], slot j % page_tok.  Inside a page a
// layer holds K as [kv head][slot][dim] and V transposed, [kv head][dim][slot].
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

#include "rg_device.h"
#include "rg_kernels.h"

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
                                                   int n_chunks, float* __restrict__ part_o,
                                                   float* __restrict__ part_ml, const int* __restrict__ d_rows) {
  const int r = blockIdx.z;
  if (r >= *d_rows) return;
  const int kvh = blockIdx.y, chunk = blockIdx.x;
  const int ctx = row_pos[r] + 1;
  const int clen = att_chunk_len(ctx, n_chunks);
  const int c0 = chunk * clen;
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
  const int32_t* tab = page_tab + (int64_t)row_tab[r] * tab_stride;
  const int64_t koff = (int64_t)layer * g.layer_elems + (int64_t)kvh * g.page_tok * hd;
  const int64_t voff = (int64_t)layer * g.layer_elems + ((int64_t)n_kv + kvh) * g.page_tok * hd;   // V^T [dim][slot]

  // each thread owns output slots (h, d) = idx / hd, idx % hd for idx = tid + 256*k
  const int n_slots = (rep * hd + 255) / 256;
  float acc[ATT_MAX_REP];
#pragma unroll
  for (int k = 0; k < ATT_MAX_REP; ++k) acc[k] = 0.f;
  __syncthreads();

  for (int t0 = c0; t0 < c1; t0 += ATT_TILE) {
    const int nt = min(ATT_TILE, c1 - t0);
    // ---- scores: one token per thread
    if (tid < nt) {
      const int j = t0 + tid;
      const KV* kp = pool + (int64_t)tab[j / g.page_tok] * g.page_elems + koff + (int64_t)(j % g.page_tok) * hd;
      float dot[ATT_MAX_REP];
#pragma unroll
      for (int h = 0; h < ATT_MAX_REP; ++h) dot[h] = 0.f;
      for (int d = 0; d < hd; d += 8) {
        float kv8[8];
        load8_f32<KV>(kp + d, kv8);
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
    for (int k = 0; k < n_slots; ++k) {
      const int idx = tid + 256 * k;
      if (idx < rep * hd) {
        const int h = idx / hd, d = idx % hd;
        float a = acc[k] * s_alpha[h];
        for (int jj = 0; jj < nt; ++jj) {
          const int j = t0 + jj;
          const KV* vp = pool + (int64_t)tab[j / g.page_tok] * g.page_elems + voff + (int64_t)d * g.page_tok;
          a = fmaf(sp[h * ATT_TILE + jj], ld_f32<KV>(vp + (j % g.page_tok)), a);
        }
        acc[k] = a;
      }
    }
    __syncthreads();
  }
  // ---- write partials
  const int64_t base = ((int64_t)r * n_chunks + chunk) * n_q + kvh * rep;
  for (int k = 0; k < n_slots; ++k) {
    const int idx = tid + 256 * k;
    if (idx < rep * hd) part_o[base * hd + idx] = acc[k];
  }
  if (tid < rep) {
    part_ml[(base + tid) * 2] = s_m[tid];
    part_ml[(base + tid) * 2 + 1] = s_l[tid];
  }
}


// ---------------------------------------------------------------- MFMA path
__device__ __forceinline__ void split8(const float* v, bf16x8_t& hi, bf16x8_t& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16_t h0 = f32_to_bf16(v[2 * i]), h1 = f32_to_bf16(v[2 * i + 1]);
    const bf16_t l0 = f32_to_bf16(v[2 * i] - bf16_to_f32(h0)), l1 = f32_to_bf16(v[2 * i + 1] - bf16_to_f32(h1));
    h[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    l[i] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  hi = __builtin_bit_cast(bf16x8_t, uint4{h[0], h[1], h[2], h[3]});
  lo = __builtin_bit_cast(bf16x8_t, uint4{l[0], l[1], l[2], l[3]});
}

constexpr int ATT_MAX_CHUNK_PAGES = 1024;   // a chunk spans at most 16384 tokens
constexpr int ATT_MAX_MERGE = 1024;         // chunks per row

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Registers of one 32-token block: K fragments of both 16-token tiles and the
// V^T fragments of every 16-dim output tile.
template <int HD>
struct AttBlock {
  u32x4_t k[2][HD / 32];
  u32x4_t v[HD / 16];
};

template <int HD>
__device__ __forceinline__ void att_load(AttBlock<HD>& b, const bf16_t* __restrict__ pool, const KvGeom& g,
                                         int64_t koff, int64_t voff, const int* spg, int c0, int c1, int t0,
                                         int col, int grp) {
  // K: A-fragment row i of tile tt is token t0 + 8*(i/4) + 4*tt + (i%4), so that
  // the S^T layout leaves lane group grp holding tokens t0+8*grp .. +7
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    int tok = t0 + 8 * (col >> 2) + 4 * tt + (col & 3);
    if (tok >= c1) tok = c0;                 // keep the load in bounds; masked later
    const bf16_t* kp = pool + (int64_t)spg[(tok - c0) >> 4] * g.page_elems + koff + (int64_t)(tok & 15) * HD + 8 * grp;
#pragma unroll
    for (int kb = 0; kb < HD / 32; ++kb) b.k[tt][kb] = *reinterpret_cast<const u32x4_t*>(kp + kb * 32);
  }
  // V^T: lane reads dims (dt*16 + col), tokens t0+8*grp .. +7 (one page slot run)
  const int tv = t0 + 8 * grp;
  const int pg = spg[((tv < c1 ? tv : c0) - c0) >> 4];
  const bf16_t* vp = pool + (int64_t)pg * g.page_elems + voff + (tv & 15);
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) b.v[dt] = *reinterpret_cast<const u32x4_t*>(vp + (int64_t)(dt * 16 + col) * 16);
}

template <int HD>
__global__ __launch_bounds__(64) void k_attention_mfma(const float* __restrict__ q, int n_q, int n_kv,
                                                       const bf16_t* __restrict__ pool, KvGeom g, int layer,
                                                       const int32_t* __restrict__ page_tab, int tab_stride,
                                                       const int32_t* __restrict__ row_tab,
                                                       const int32_t* __restrict__ row_pos,
                                                       int n_chunks, int rows_ub, float* __restrict__ part_o,
                                                       float* __restrict__ part_ml, const int* __restrict__ d_rows) {
  static_assert(HD % 32 == 0 && HD <= 256, "head_dim");
  // XCD-aware order: the 1-D grid has a multiple of 8 blocks and blocks are
  // dealt to the 8 XCDs round-robin, so XCD x = b % 8 takes the contiguous
  // work range [x*per_xcd, (x+1)*per_xcd): neighbouring rows (siblings of one
  // prompt) share an XCD, whose L2 then holds their shared prefix.
  const int64_t nb = (int64_t)n_chunks * n_kv * rows_ub;
  const int64_t b = blockIdx.x;
  const int64_t per_xcd = (int64_t)gridDim.x / 8;
  const int64_t w = (b % 8) * per_xcd + b / 8;
  if (w >= nb) return;
  const int chunk = (int)(w % n_chunks);
  const int kvh = (int)((w / n_chunks) % n_kv);
  const int r = (int)(w / ((int64_t)n_chunks * n_kv));
  if (r >= *d_rows) return;
  const int ctx = row_pos[r] + 1;
  const int clen = att_chunk_len(ctx, n_chunks);
  const int c0 = chunk * clen;
  if (c0 >= ctx) return;
  const int c1 = min(ctx, c0 + clen);
  const int rep = n_q / n_kv;
  const int lane = threadIdx.x, col = lane & 15, grp = lane >> 4;

  // page ids of the chunk, once
  __shared__ int spg[ATT_MAX_CHUNK_PAGES];
  {
    const int32_t* tab = page_tab + (int64_t)row_tab[r] * tab_stride + (c0 >> 4);
    const int npg = (c1 - c0 + 15) >> 4;
    for (int i = lane; i < npg; i += 64) spg[i] = tab[i];
    __syncthreads();
  }
  // Q^T fragments: lane holds q[head col][kb*32 + 8*grp + 0..7], pre-scaled by 1/sqrt(hd)
  bf16x8_t qh[HD / 32], ql[HD / 32];
  {
    const float scale = 1.0f / sqrtf((float)HD);
    const float* qr = q + ((int64_t)r * n_q + kvh * rep + min(col, rep - 1)) * HD + 8 * grp;   // lanes >= rep: padding
#pragma unroll
    for (int kb = 0; kb < HD / 32; ++kb) {
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = col < rep ? qr[kb * 32 + i] * scale : 0.f;
      split8(v, qh[kb], ql[kb]);
    }
  }
  const int64_t koff = (int64_t)layer * g.layer_elems + (int64_t)kvh * 16 * HD;
  const int64_t voff = (int64_t)layer * g.layer_elems + ((int64_t)n_kv + kvh) * 16 * HD;

  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t oacc[HD / 16];
#pragma unroll
  for (int i = 0; i < HD / 16; ++i) oacc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  AttBlock<HD> cur, nxt;
  att_load<HD>(cur, pool, g, koff, voff, spg, c0, c1, c0, col, grp);
  for (int t0 = c0; t0 < c1; t0 += 32) {
    if (t0 + 32 < c1) att_load<HD>(nxt, pool, g, koff, voff, spg, c0, c1, t0 + 32, col, grp);   // next block in flight
    // ---- S^T = K Q^T; lane holds tokens t0 + 8*grp + 4*tt + j of query head col
    f32x4_t s[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < HD / 32; ++kb) {
        const bf16x8_t kf = __builtin_bit_cast(bf16x8_t, cur.k[tt][kb]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qh[kb], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, ql[kb], acc, 0, 0, 0);
      }
      s[tt] = acc;
    }
    const int nval = min(8, max(0, c1 - (t0 + 8 * grp)));   // valid tokens among this lane group's 8
    float mloc = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (4 * tt + j >= nval) s[tt][j] = -INFINITY;
        mloc = fmaxf(mloc, s[tt][j]);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_run, mloc);
    const float alpha = expf(m_run - m_new);       // 0 on the first block
    float p[8];
    float psum = 0.f;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float e = expf(s[tt][j] - m_new);    // exp(-inf) = 0 for masked tokens
        p[tt * 4 + j] = e;
        psum += e;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < HD / 16; ++i) oacc[i] *= alpha;
    bf16x8_t ph, pl;
    split8(p, ph, pl);
    // ---- O^T += V^T P^T (k = this lane group's 8 tokens, in order)
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      u32x4_t vv = cur.v[dt];
      if (nval < 8) {   // zero the slots of masked tokens (their memory may hold anything)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int n2 = nval - 2 * e;   // valid tokens in this dword
          vv[e] = n2 >= 2 ? vv[e] : (n2 == 1 ? (vv[e] & 0xFFFFu) : 0u);
        }
      }
      const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, vv);
      oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, ph, oacc[dt], 0, 0, 0);
      oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl, oacc[dt], 0, 0, 0);
    }
    cur = nxt;
  }
  // ---- partials: lane holds O^T[dims dt*16 + 4*grp + j][head col]
  if (col < rep) {
    const int64_t base = ((int64_t)r * n_chunks + chunk) * n_q + kvh * rep + col;
    float* po = part_o + base * HD;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) po[dt * 16 + 4 * grp + j] = oacc[dt][j];
    if (grp == 0) {
      part_ml[base * 2] = m_run;
      part_ml[base * 2 + 1] = l_run;
    }
  }
}

template <int SPLIT>
__global__ void k_attn_merge(const float* __restrict__ part_o, const float* __restrict__ part_ml, int n_q, int hd,
                             const int32_t* __restrict__ row_pos, int n_chunks, ActOut out,
                             const int* __restrict__ d_rows) {
  const int r = blockIdx.x;
  if (r >= *d_rows) return;
  const int h = blockIdx.y;
  const int ctx = row_pos[r] + 1;
  const int clen = att_chunk_len(ctx, n_chunks);
  const int nc = (ctx + clen - 1) / clen;   // chunks holding context
  __shared__ float sw[ATT_MAX_MERGE];       // chunk weights exp(m_c - M) / L
  // (max, sum) of every chunk: one thread per chunk, then a wave reduction
  const int64_t rb = (int64_t)r * n_chunks;
  float m = -INFINITY;
  for (int c = threadIdx.x; c < nc; c += blockDim.x) m = fmaxf(m, part_ml[((rb + c) * n_q + h) * 2]);
  __shared__ float red[16];
  const float M = block_max(m, red);
  float l = 0.f;
  for (int c = threadIdx.x; c < nc; c += blockDim.x) {
    const float* ml = part_ml + ((rb + c) * n_q + h) * 2;
    const float w = expf(ml[0] - M);
    sw[c] = w;
    l += w * ml[1];
  }
  const float invL = 1.0f / block_sum(l, red);
  for (int d = threadIdx.x; d < hd; d += blockDim.x) {
    float o0 = 0.f, o1 = 0.f, o2 = 0.f, o3 = 0.f;   // independent sums keep several loads in flight
    int c = 0;
    for (; c + 4 <= nc; c += 4) {
      o0 += sw[c] * part_o[((rb + c) * n_q + h) * hd + d];
      o1 += sw[c + 1] * part_o[((rb + c + 1) * n_q + h) * hd + d];
      o2 += sw[c + 2] * part_o[((rb + c + 2) * n_q + h) * hd + d];
      o3 += sw[c + 3] * part_o[((rb + c + 3) * n_q + h) * hd + d];
    }
    for (; c < nc; ++c) o0 += sw[c] * part_o[((rb + c) * n_q + h) * hd + d];
    act_store<SPLIT>(out, ((int64_t)r * n_q + h) * hd + d, ((o0 + o1) + (o2 + o3)) * invL);
  }
}

}  // namespace

hipError_t launch_attention(int dtype, const float* q, int n_q, int n_kv, int head_dim, const void* kv_pool,
                            KvGeom g, int layer, const int32_t* page_tab, int tab_stride,
                            const int32_t* row_tab, const int32_t* row_pos, int max_ctx, int n_chunks,
                            float* part_o, float* part_ml, const int* d_rows, int rows_ub, hipStream_t st) {
  if (n_chunks < 1 || n_chunks > ATT_MAX_MERGE ||
      std::max(128, (max_ctx + n_chunks - 1) / n_chunks + 31) > 16 * ATT_MAX_CHUNK_PAGES)
    return hipErrorInvalidValue;
  if (rows_ub <= 0) return hipSuccess;
  dim3 grid(n_chunks, n_kv, rows_ub);
  if (dtype == 1) {
    // two 16-slot pages per 32-token block
    if (g.page_tok != 16) return hipErrorInvalidValue;
    const int64_t nb = (int64_t)n_chunks * n_kv * rows_ub;
    const dim3 grid1((unsigned)((nb + 7) / 8 * 8));
#define RG_ATT_MFMA(HD)                                                                                          \
    hipLaunchKernelGGL(k_attention_mfma<HD>, grid1, dim3(64), 0, st, q, n_q, n_kv, (const bf16_t*)kv_pool, g, layer, \
                       page_tab, tab_stride, row_tab, row_pos, n_chunks, rows_ub, part_o, part_ml, d_rows)
    switch (head_dim) {
      case 64: RG_ATT_MFMA(64); break;
      case 128: RG_ATT_MFMA(128); break;
      default: return hipErrorInvalidValue;
    }
#undef RG_ATT_MFMA
  } else
    hipLaunchKernelGGL(k_attention<float>, grid, dim3(256), 0, st, q, n_q, n_kv, head_dim, (const float*)kv_pool,
                       g, layer, page_tab, tab_stride, row_tab, row_pos, n_chunks, part_o, part_ml, d_rows);
  return hipGetLastError();
}

hipError_t launch_attn_merge(int dtype, const float* part_o, const float* part_ml, int n_q, int head_dim,
                             const int32_t* row_pos, int n_chunks, void* out, int64_t a_plane,
                             const int* d_rows, int rows_ub, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  if (n_chunks < 1 || n_chunks > ATT_MAX_MERGE) return hipErrorInvalidValue;
  dim3 grid(rows_ub, n_q);
  int threads = head_dim >= 64 ? 64 * ((head_dim + 63) / 64) : 64;
  const ActOut o{out, a_plane};
  if (dtype == 1)
    hipLaunchKernelGGL(k_attn_merge<1>, grid, dim3(threads), 0, st, part_o, part_ml, n_q, head_dim, row_pos,
                       n_chunks, o, d_rows);
  else
    hipLaunchKernelGGL(k_attn_merge<0>, grid, dim3(threads), 0, st, part_o, part_ml, n_q, head_dim, row_pos,
                       n_chunks, o, d_rows);
  return hipGetLastError();
}
