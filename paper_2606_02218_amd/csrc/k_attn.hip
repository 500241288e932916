// Paged causal attention over the KV pool, for prefill rows and decode rows
// alike.  Each block handles (row, kv head, chunk of the row's context): it
// scores up to 256 context tokens per tile against the GQA group's query heads
// (fp32, keys/values converted from the storage type), keeps a running
// softmax (max, sum) and accumulates the unnormalised output; the merge kernel
// combines the chunks.  Context positions 0..row_pos[r] of page table
// row_tab[r]; position j lives in page page_tab[tab*tab_stride + j/page_tok],
// slot j % page_tok.
#include "rg_device.h"
#include "rg_kernels.h"

namespace {

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
                                                   const int32_t* __restrict__ row_pos, int chunk_len,
                                                   int n_chunks, float* __restrict__ part_o,
                                                   float* __restrict__ part_ml, const int* __restrict__ d_rows) {
  const int r = blockIdx.z;
  if (r >= *d_rows) return;
  const int kvh = blockIdx.y, chunk = blockIdx.x;
  const int ctx = row_pos[r] + 1;
  const int c0 = chunk * chunk_len;
  if (c0 >= ctx) return;
  const int c1 = min(ctx, c0 + chunk_len);
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
  const int64_t voff = koff + (int64_t)n_kv * g.page_tok * hd;

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
          const KV* vp = pool + (int64_t)tab[j / g.page_tok] * g.page_elems + voff + (int64_t)(j % g.page_tok) * hd;
          a = fmaf(sp[h * ATT_TILE + jj], ld_f32<KV>(vp + d), a);
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

template <int SPLIT>
__global__ void k_attn_merge(const float* __restrict__ part_o, const float* __restrict__ part_ml, int n_q, int hd,
                             const int32_t* __restrict__ row_pos, int chunk_len, int n_chunks, ActOut out,
                             const int* __restrict__ d_rows) {
  const int r = blockIdx.x;
  if (r >= *d_rows) return;
  const int h = blockIdx.y;
  const int nc = (row_pos[r] + chunk_len) / chunk_len;   // chunks holding context
  float M = -INFINITY;
  for (int c = 0; c < nc; ++c) M = fmaxf(M, part_ml[(((int64_t)r * n_chunks + c) * n_q + h) * 2]);
  float L = 0.f;
  for (int c = 0; c < nc; ++c) {
    const float* ml = part_ml + (((int64_t)r * n_chunks + c) * n_q + h) * 2;
    L += expf(ml[0] - M) * ml[1];
  }
  const float invL = 1.0f / L;
  for (int d = threadIdx.x; d < hd; d += blockDim.x) {
    float o = 0.f;
    for (int c = 0; c < nc; ++c) {
      const int64_t b = ((int64_t)r * n_chunks + c) * n_q + h;
      o += expf(part_ml[b * 2] - M) * part_o[b * hd + d];
    }
    act_store<SPLIT>(out, ((int64_t)r * n_q + h) * hd + d, o * invL);
  }
}

}  // namespace

hipError_t launch_attention(int dtype, const float* q, int n_q, int n_kv, int head_dim, const void* kv_pool,
                            KvGeom g, int layer, const int32_t* page_tab, int tab_stride,
                            const int32_t* row_tab, const int32_t* row_pos, int chunk_len, int n_chunks,
                            float* part_o, float* part_ml, const int* d_rows, int rows_ub, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  dim3 grid(n_chunks, n_kv, rows_ub);
  if (dtype == 1)
    hipLaunchKernelGGL(k_attention<bf16_t>, grid, dim3(256), 0, st, q, n_q, n_kv, head_dim, (const bf16_t*)kv_pool,
                       g, layer, page_tab, tab_stride, row_tab, row_pos, chunk_len, n_chunks, part_o, part_ml,
                       d_rows);
  else
    hipLaunchKernelGGL(k_attention<float>, grid, dim3(256), 0, st, q, n_q, n_kv, head_dim, (const float*)kv_pool,
                       g, layer, page_tab, tab_stride, row_tab, row_pos, chunk_len, n_chunks, part_o, part_ml,
                       d_rows);
  return hipGetLastError();
}

hipError_t launch_attn_merge(int dtype, const float* part_o, const float* part_ml, int n_q, int head_dim,
                             const int32_t* row_pos, int chunk_len, int n_chunks, void* out, int64_t a_plane,
                             const int* d_rows, int rows_ub, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  dim3 grid(rows_ub, n_q);
  int threads = head_dim >= 64 ? 64 * ((head_dim + 63) / 64) : 64;
  const ActOut o{out, a_plane};
  if (dtype == 1)
    hipLaunchKernelGGL(k_attn_merge<1>, grid, dim3(threads), 0, st, part_o, part_ml, n_q, head_dim, row_pos,
                       chunk_len, n_chunks, o, d_rows);
  else
    hipLaunchKernelGGL(k_attn_merge<0>, grid, dim3(threads), 0, st, part_o, part_ml, n_q, head_dim, row_pos,
                       chunk_len, n_chunks, o, d_rows);
  return hipGetLastError();
}
