// Row-wise kernels of the decoder step: embedding gather and row set-up,
// RMSNorm, residual add, page copies, plus the Philox test hooks.
#include "rg_device.h"
#include "rg_kernels.h"

namespace {

template <typename T>
__global__ void k_embed(const T* __restrict__ embed, int d, int V, const int32_t* __restrict__ tok,
                        float* __restrict__ x, int32_t* __restrict__ bad_token, const int* __restrict__ d_rows) {
  const int r = blockIdx.x;
  if (r >= *d_rows) return;
  int id = tok[r];
  if (id < 0 || id >= V) {
    if (threadIdx.x == 0) bad_token[0] = 1;
    id = 0;
  }
  const T* e = embed + (int64_t)id * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(int64_t)r * d + i] = ld_f32<T>(e + i);
}

template <typename T>
__global__ void k_decode_rows(const T* __restrict__ embed, int d, const int32_t* __restrict__ act_seq,
                              const int32_t* __restrict__ act_tok, const int32_t* __restrict__ seq_grp,
                              const int32_t* __restrict__ plen, const int* __restrict__ d_t, int prefix_split,
                              int32_t* __restrict__ row_tab, int32_t* __restrict__ row_pos,
                              int32_t* __restrict__ row_beg, float* __restrict__ x, const int* __restrict__ d_rows) {
  const int r = blockIdx.x;
  if (r >= *d_rows) return;
  const int s = act_seq[r];
  if (threadIdx.x == 0) {
    const int L = plen[seq_grp[s]];
    row_tab[r] = s;
    row_pos[r] = L + *d_t - 1;
    row_beg[r] = prefix_split ? (L >> 4) << 4 : 0;
  }
  const T* e = embed + (int64_t)act_tok[r] * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(int64_t)r * d + i] = ld_f32<T>(e + i);
}

__global__ void k_prefill_rows(const int32_t* __restrict__ prompt_off, int P, int tab_base,
                               int32_t* __restrict__ row_tab, int32_t* __restrict__ row_pos,
                               int32_t* __restrict__ row_beg, int total) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= total) return;
  int lo = 0, hi = P - 1;   // last p with prompt_off[p] <= r
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (prompt_off[mid] <= r) lo = mid; else hi = mid - 1;
  }
  row_tab[r] = tab_base + lo;
  row_pos[r] = r - prompt_off[lo];
  row_beg[r] = 0;
}

// Streaming ceiling of the memory system (a measurement aid for the
// rooflines, not a step of the path): each thread reads eight 16-byte pieces
// per iteration of a grid-stride loop, one grid-stride apart, so every wave
// reads whole contiguous 1 KB runs, with non-temporal loads (and stores)
// that do not claim cache space.  MODE 1 writes them to dst (a copy); MODE 0
// folds them into one word per thread, stored to sink, so the loads stay
// live (a read).
typedef uint32_t probe_u32x4 __attribute__((ext_vector_type(4)));
template <int MODE>
__global__ __launch_bounds__(256) void k_hbm_probe(const probe_u32x4* __restrict__ src, probe_u32x4* __restrict__ dst,
                                                   int64_t n16, uint32_t* __restrict__ sink) {
  constexpr int U = 8;
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    probe_u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(&src[i + u * stride]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if constexpr (MODE == 1) __builtin_nontemporal_store(v[u], &dst[i + u * stride]);
      else acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
  }
  for (; i < n16; i += stride) {
    const probe_u32x4 v = __builtin_nontemporal_load(&src[i]);
    if constexpr (MODE == 1) __builtin_nontemporal_store(v, &dst[i]);
    else acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if constexpr (MODE == 0) sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

template <int SPLIT>
__global__ __launch_bounds__(256) void k_rmsnorm(const float* __restrict__ x, const float* __restrict__ g, int d,
                                                 float eps, ActOut out, const int32_t* __restrict__ src_rows,
                                                 const int* __restrict__ d_rows) {
  const int r = blockIdx.x;
  if (r >= *d_rows) return;
  __shared__ float red[16];
  const float* xr = x + (int64_t)(src_rows ? src_rows[r] : r) * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += blockDim.x) ss = fmaf(xr[i], xr[i], ss);
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += blockDim.x) act_store<SPLIT>(out, (int64_t)r * d + i, xr[i] * inv * g[i]);
}

// Copy-on-write of whole pages: every layer's slab of page pairs[2k] to page
// pairs[2k+1], for k < state[3].
template <typename KV>
__global__ void k_page_copy(KV* __restrict__ pool, KvGeom g, const int32_t* __restrict__ pairs,
                            const int32_t* __restrict__ state) {
  const int k = blockIdx.y;
  if (k >= state[3]) return;
  const int64_t src = (int64_t)pairs[2 * k] * g.page_stride, dst = (int64_t)pairs[2 * k + 1] * g.page_stride;
  const int64_t n = g.slab_elems * g.n_layers;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t l = i / g.slab_elems, j = i - l * g.slab_elems;
    pool[dst + l * g.layer_stride + j] = pool[src + l * g.layer_stride + j];
  }
}

__global__ void k_fill_i32(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

__global__ void k_philox_blocks(uint64_t k0, uint64_t k1, const uint64_t* __restrict__ ctr, int64_t n,
                                uint64_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  rg_u64x4 c;
#pragma unroll
  for (int j = 0; j < 4; ++j) c.v[j] = ctr[4 * i + j];
  rg_u64x4 o = rg_philox4x64_10(c, k0, k1);
#pragma unroll
  for (int j = 0; j < 4; ++j) out[4 * i + j] = o.v[j];
}

__global__ void k_gumbel_bits(uint64_t seed, int t, int s, int vocab, uint32_t* __restrict__ out) {
  const int vb = blockIdx.x * blockDim.x + threadIdx.x;
  if (vb * 8 >= vocab) return;
  rg_u64x4 c;
  c.v[0] = (uint64_t)vb; c.v[1] = (uint64_t)t; c.v[2] = (uint64_t)s; c.v[3] = 0;
  rg_u64x4 w = rg_philox4x64_10(c, seed, RG_TAG_GUMBEL);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int v = vb * 8 + j;
    if (v < vocab) out[v] = (uint32_t)(w.v[j >> 1] >> (32 * (j & 1)));
  }
}

}  // namespace


hipError_t launch_embed(int dtype, const void* embed, int d, int V, const int32_t* tok, float* x, int32_t* bad_token,
                        const int* d_rows, int rows_ub, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(k_embed<bf16_t>, dim3(rows_ub), dim3(256), 0, st, (const bf16_t*)embed, d, V, tok, x, bad_token,
                       d_rows);
  else
    hipLaunchKernelGGL(k_embed<float>, dim3(rows_ub), dim3(256), 0, st, (const float*)embed, d, V, tok, x, bad_token,
                       d_rows);
  return hipGetLastError();
}

hipError_t launch_decode_rows(int dtype, const void* embed, int d, const int32_t* act_seq, const int32_t* act_tok,
                              const int32_t* seq_grp, const int32_t* plen, const int* d_t, int prefix_split,
                              int32_t* row_tab, int32_t* row_pos, int32_t* row_beg, float* x, const int* d_rows,
                              int rows_ub, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(k_decode_rows<bf16_t>, dim3(rows_ub), dim3(256), 0, st, (const bf16_t*)embed, d, act_seq, act_tok,
                       seq_grp, plen, d_t, prefix_split, row_tab, row_pos, row_beg, x, d_rows);
  else
    hipLaunchKernelGGL(k_decode_rows<float>, dim3(rows_ub), dim3(256), 0, st, (const float*)embed, d, act_seq, act_tok,
                       seq_grp, plen, d_t, prefix_split, row_tab, row_pos, row_beg, x, d_rows);
  return hipGetLastError();
}

hipError_t launch_prefill_rows(const int32_t* prompt_off, int P, int tab_base, int32_t* row_tab, int32_t* row_pos,
                               int32_t* row_beg, int total, hipStream_t st) {
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_prefill_rows, dim3((total + 255) / 256), dim3(256), 0, st, prompt_off, P, tab_base, row_tab,
                     row_pos, row_beg, total);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, const float* x, const float* g, int d, float eps, void* out, int64_t a_plane,
                          const int32_t* src_rows, const int* d_rows, int rows_ub, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  const ActOut o{out, a_plane};
  if (dtype == 1)
    hipLaunchKernelGGL(k_rmsnorm<1>, dim3(rows_ub), dim3(256), 0, st, x, g, d, eps, o, src_rows, d_rows);
  else
    hipLaunchKernelGGL(k_rmsnorm<0>, dim3(rows_ub), dim3(256), 0, st, x, g, d, eps, o, src_rows, d_rows);
  return hipGetLastError();
}

hipError_t launch_page_copy(int dtype, void* kv_pool, const KvGeom& g, const int32_t* copy_pairs, int max_pairs,
                            const int32_t* state, hipStream_t st) {
  if (max_pairs <= 0) return hipSuccess;
  dim3 grid(64, max_pairs);
  if (dtype == 1)
    hipLaunchKernelGGL(k_page_copy<bf16_t>, grid, dim3(256), 0, st, (bf16_t*)kv_pool, g, copy_pairs, state);
  else
    hipLaunchKernelGGL(k_page_copy<float>, grid, dim3(256), 0, st, (float*)kv_pool, g, copy_pairs, state);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)blocks), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_philox_blocks(uint64_t k0, uint64_t k1, const uint64_t* ctr, int64_t n, uint64_t* out,
                                hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_philox_blocks, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, k0, k1, ctr, n, out);
  return hipGetLastError();
}

hipError_t launch_gumbel_bits(uint64_t seed, int t, int s, int vocab, uint32_t* out, hipStream_t st) {
  const int nb = (vocab + 7) / 8;
  hipLaunchKernelGGL(k_gumbel_bits, dim3((nb + 255) / 256), dim3(256), 0, st, seed, t, s, vocab, out);
  return hipGetLastError();
}

hipError_t launch_hbm_probe(const void* src, void* dst, int64_t bytes, int mode, int blocks, hipStream_t st) {
  if (bytes <= 0) return hipSuccess;
  const int64_t n16 = bytes / 16;
  if (mode == 1)
    hipLaunchKernelGGL(k_hbm_probe<1>, dim3(blocks), dim3(256), 0, st, (const probe_u32x4*)src, (probe_u32x4*)dst, n16,
                       nullptr);
  else
    hipLaunchKernelGGL(k_hbm_probe<0>, dim3(blocks), dim3(256), 0, st, (const probe_u32x4*)src, nullptr, n16,
                       (uint32_t*)dst);
  return hipGetLastError();
}
