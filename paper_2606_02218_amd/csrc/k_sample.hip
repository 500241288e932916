// Token sampling, retirement/compaction, sibling fork, rollout set-up and the
// group-relative advantage.
#include "rg_device.h"
#include "rg_kernels.h"

namespace {

// ------------------------------------------------------------------ sampling
// Two kernels.  k_sample_slice: block (slice, row) scans one slice of the
// row's vocabulary -- Gumbel scores, running logsumexp of z/T -- and writes
// the slice's (best score, best id, max, sum).  k_sample_pick: one block per
// row combines the slices in order (ties to the lowest id), decides the
// token and writes the outputs.
constexpr int SAMPLE_THREADS = 256;

__global__ __launch_bounds__(SAMPLE_THREADS) void k_sample_slice(SampleArgs a) {
  const int r = blockIdx.y;
  if (r >= *a.d_rows) return;
  const int tid = threadIdx.x;
  const int t = *a.d_t;
  const int s = a.act_seq[r];
  const int lrow = a.logits_by_group ? a.seq_grp[s] : r;
  const float* z = a.logits + (int64_t)lrow * a.V;
  const int L = a.forced_len ? a.forced_len[s] : -1;
  const bool mask_eos = L > 0 && t < L - 1;
  const float T = a.temperature;
  const bool unit_T = T == 1.0f;                            // z / 1 == z exactly: skip the division
  const int nb = a.V >> 3;                                  // 8-token Philox blocks
  const int per = (nb + a.n_slices - 1) / a.n_slices;
  const int vb0 = blockIdx.x * per, vb1 = min(nb, vb0 + per);

  // the EOS entry is masked in one 8-token block only
  const int eos_vb = mask_eos ? (a.eos >> 3) : -1, eos_j = a.eos & 7;
  float best = -INFINITY;
  int best_v = 0x7FFFFFFF;
  float m = -INFINITY, sum = 0.f;
  for (int vb = vb0 + tid; vb < vb1; vb += SAMPLE_THREADS) {
    rg_u64x4 c;
    c.v[0] = (uint64_t)vb; c.v[1] = (uint64_t)t; c.v[2] = (uint64_t)s; c.v[3] = 0;
    rg_u64x4 w = rg_philox4x64_10(c, a.seed, RG_TAG_GUMBEL);
    const float4 z0 = *reinterpret_cast<const float4*>(z + vb * 8);
    const float4 z1 = *reinterpret_cast<const float4*>(z + vb * 8 + 4);
    float zt[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
    if (!unit_T) {
#pragma unroll
      for (int j = 0; j < 8; ++j) zt[j] /= T;                // z / 1 == z exactly: skipped at T = 1
    }
    // running logsumexp, rescaled once per 8 tokens (hardware exponential,
    // relative error ~1e-7)
    float bm = zt[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) bm = fmaxf(bm, zt[j]);
    if (bm > m) { sum *= __expf(m - bm); m = bm; }
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += __expf(zt[j] - m);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t bits = (uint32_t)(w.v[j >> 1] >> (32 * (j & 1)));
      const float u = rg_uniform_from_bits(bits);
      // Gumbel noise -log(-log u): the inner log keeps full accuracy (for u
      // near 1 its result is ~6e-8, where only a relative-error log is safe);
      // the outer one takes an argument in [6e-8, 16.7] and needs ~1e-7
      // absolute accuracy, which the hardware logarithm gives
      float sc = zt[j] + (-__logf(-logf(u)));
      if (vb == eos_vb && j == eos_j) sc = -INFINITY;
      // a thread scans increasing ids, so a strict > keeps the lowest id of a tie
      if (sc > best) { best = sc; best_v = vb * 8 + j; }
    }
    if (a.dump_logits && t < a.dump_steps) {
      float* dst = a.dump_logits + ((int64_t)t * a.n_seq + s) * a.V + vb * 8;
      *reinterpret_cast<float4*>(dst) = z0;
      *reinterpret_cast<float4*>(dst + 4) = z1;
    }
  }
  __shared__ float sb[SAMPLE_THREADS], sm[SAMPLE_THREADS], ss[SAMPLE_THREADS];
  __shared__ int sv[SAMPLE_THREADS];
  sb[tid] = best; sv[tid] = best_v; sm[tid] = m; ss[tid] = sum;
  __syncthreads();
  for (int o = SAMPLE_THREADS / 2; o > 0; o >>= 1) {
    if (tid < o) {
      const float b2 = sb[tid + o]; const int v2 = sv[tid + o];
      if (b2 > sb[tid] || (b2 == sb[tid] && v2 < sv[tid])) { sb[tid] = b2; sv[tid] = v2; }
      const float m1 = sm[tid], m2 = sm[tid + o];
      const float mm = fmaxf(m1, m2);
      ss[tid] = (m1 == -INFINITY ? 0.f : ss[tid] * expf(m1 - mm)) + (m2 == -INFINITY ? 0.f : ss[tid + o] * expf(m2 - mm));
      sm[tid] = mm;
    }
    __syncthreads();
  }
  if (tid == 0) {
    float* p = a.part + ((int64_t)r * a.n_slices + blockIdx.x) * 4;
    p[0] = sb[0];
    p[1] = __int_as_float(sv[0]);
    p[2] = sm[0];
    p[3] = ss[0];
  }
}

// One wave per row: lane l combines slices l, l + 64, ... in order, then the
// lanes' results are combined across the wave (best score, ties to the
// lowest id; logsumexp by max and rescaled sums).
__global__ __launch_bounds__(64) void k_sample_pick(SampleArgs a) {
  const int r = blockIdx.x;
  if (r >= *a.d_rows) return;
  const int lane = threadIdx.x;
  float best = -INFINITY, m = -INFINITY, sum = 0.f;
  int y = 0x7FFFFFFF;
  for (int k = lane; k < a.n_slices; k += 64) {
    const float4 p = *reinterpret_cast<const float4*>(a.part + ((int64_t)r * a.n_slices + k) * 4);
    const int v2 = __float_as_int(p.y);
    if (p.x > best || (p.x == best && v2 < y)) { best = p.x; y = v2; }
    const float mm = fmaxf(m, p.z);
    sum = (m == -INFINITY ? 0.f : sum * expf(m - mm)) + (p.z == -INFINITY ? 0.f : p.w * expf(p.z - mm));
    m = mm;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float b2 = __shfl_xor(best, o, 64), m2 = __shfl_xor(m, o, 64), s2 = __shfl_xor(sum, o, 64);
    const int v2 = __shfl_xor(y, o, 64);
    if (b2 > best || (b2 == best && v2 < y)) { best = b2; y = v2; }
    const float mm = fmaxf(m, m2);
    sum = (m == -INFINITY ? 0.f : sum * expf(m - mm)) + (m2 == -INFINITY ? 0.f : s2 * expf(m2 - mm));
    m = mm;
  }
  if (lane != 0) return;
  const int t = *a.d_t;
  const int s = a.act_seq[r];
  const int lrow = a.logits_by_group ? a.seq_grp[s] : r;
  const float* z = a.logits + (int64_t)lrow * a.V;
  const int L = a.forced_len ? a.forced_len[s] : -1;
  if (L > 0 && t == L - 1) y = a.eos;
  int fed = a.force_tokens ? a.force_tokens[(int64_t)s * a.max_new + t] : y;
  if (fed < 0 || fed >= a.V) { fed = a.eos; a.bad_token[0] = 1; }   // invalid forced id: stop this sequence
  const float lse = m + logf(sum);
  const float lp = z[fed] / a.temperature - lse;
  a.tokens_out[(int64_t)s * a.max_new + t] = y;
  a.logprobs_out[(int64_t)s * a.max_new + t] = lp;
  a.next_tok[r] = fed;
  a.done[r] = (fed == a.eos || t + 1 == a.max_new) ? 1 : 0;
}

// ------------------------------------------------------------------ retirement
// One block.  Pass 1 retires finished rows (length, private pages back to the
// free stack); pass 2 compacts the surviving rows in place (stable) and gives
// each survivor whose next position starts a page a fresh page.
__global__ __launch_bounds__(1024) void k_compact(CompactArgs a) {
  __shared__ int lds[17];
  __shared__ unsigned long long s_ctx;
  __shared__ int s_groups;
  const int tid = threadIdx.x;
  const int M = a.state[0];
  const int t = a.state[8];
  int top = a.state[1];
  if (tid == 0) { s_ctx = 0; s_groups = 0; }
  __syncthreads();
  // pass 1
  int carry = 0;
  for (int base = 0; base < M; base += blockDim.x) {
    const int r = base + tid;
    int f = 0, s = -1;
    bool dn = false;
    if (r < M) {
      s = a.act_seq[r];
      dn = a.done[r] != 0;
      const int p = a.seq_grp[s];
      atomicAdd(&s_ctx, (unsigned long long)a.plen[p]);
      if (r == 0 || a.seq_grp[a.act_seq[r - 1]] != p) atomicAdd(&s_groups, 1);
      if (dn) f = a.seq_npages[s] - a.seq_nshared[s];
    }
    int tot;
    const int off = block_excl_scan(f, lds, &tot) + carry;
    if (dn) {
      a.lengths[s] = t + 1;
      const int32_t* tab = a.page_tab + (int64_t)s * a.max_pages + a.seq_nshared[s];
      for (int i = 0; i < f; ++i) a.free_stack[top + off + i] = tab[i];
      a.seq_npages[s] = a.seq_nshared[s];
    }
    carry += tot;
  }
  top += carry;
  __syncthreads();
  // pass 2
  int kcarry = 0, ncarry = 0;
  bool oom = false;
  for (int base = 0; base < M; base += blockDim.x) {
    const int r = base + tid;
    int s = -1, tok = 0, keep = 0, need = 0;
    if (r < M) {
      s = a.act_seq[r];
      tok = a.act_tok[r];
      keep = a.done[r] == 0;
      need = keep && ((a.plen[a.seq_grp[s]] + t) % a.page_tok == 0);
    }
    __syncthreads();   // every read of this tile precedes any in-place write
    int ktot, ntot;
    const int kidx = block_excl_scan(keep, lds, &ktot) + kcarry;
    const int nidx = block_excl_scan(need, lds, &ntot) + ncarry;
    if (keep) { a.act_seq[kidx] = s; a.act_tok[kidx] = tok; }
    if (need) {
      const int slot = top - 1 - nidx;
      const int np = a.seq_npages[s];
      if (slot >= 0 && np < a.max_pages) {
        a.page_tab[(int64_t)s * a.max_pages + np] = a.free_stack[slot];
        a.seq_npages[s] = np + 1;
      }
    }
    kcarry += ktot;
    ncarry += ntot;
  }
  if (ncarry > top) oom = true;
  // pass 3: row range of every prompt among the kept rows (in sequence
  // order, so each prompt's rows are contiguous)
  const int M2 = oom ? 0 : kcarry;
  for (int p = tid; p < a.P; p += blockDim.x) { a.grp_row0[p] = 0; a.grp_row1[p] = 0; }
  __syncthreads();   // the resets and the compacted act_seq precede the range writes
  for (int r = tid; r < M2; r += blockDim.x) {
    const int p = a.seq_grp[a.act_seq[r]];
    if (r == 0 || a.seq_grp[a.act_seq[r - 1]] != p) a.grp_row0[p] = r;
    if (r == M2 - 1 || a.seq_grp[a.act_seq[r + 1]] != p) a.grp_row1[p] = r + 1;
  }
  if (tid == 0) {
    if (t < a.hist_cap) {
      a.hist_active[t] = M;
      a.hist_groups[t] = s_groups;
      a.hist_ctx[t] = (int64_t)s_ctx;
    }
    if (oom) { a.state[2] = 1; a.state[0] = 0; }
    else { a.state[0] = kcarry; a.state[1] = top - ncarry; }
    a.state[8] = t + 1;   // the next step
  }
}

// ------------------------------------------------------------------ fork
// One block.  Sequence s (prompt p, sibling j) gets the prompt's full pages
// by reference (shared) and private copies of the rest: the partial last
// page, or every page when sharing is off.
__global__ __launch_bounds__(1024) void k_fork(ForkArgs a) {
  __shared__ int lds[17];
  const int tid = threadIdx.x;
  int top = a.state[1];
  int carry = 0;
  for (int base = 0; base < a.n_seq; base += blockDim.x) {
    const int s = base + tid;
    int need = 0, p = 0, n_pref = 0, shared = 0;
    if (s < a.n_seq) {
      int lo = 0, hi = a.P - 1;   // last p with grp_off[p] <= s
      while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (a.grp_off[mid] <= s) lo = mid; else hi = mid - 1;
      }
      p = lo;
      const int L = a.plen[p];
      const int n_full = L / a.page_tok;
      n_pref = (L + a.page_tok - 1) / a.page_tok;
      shared = a.share ? n_full : 0;
      need = n_pref - shared;
    }
    int tot;
    const int off = block_excl_scan(need, lds, &tot) + carry;
    if (s < a.n_seq) {
      a.seq_grp[s] = p;
      a.act_seq[s] = s;
      a.seq_npages[s] = n_pref;
      a.seq_nshared[s] = shared;
      const int32_t* ptab = a.page_tab + (int64_t)(a.n_seq + p) * a.max_pages;
      int32_t* stab = a.page_tab + (int64_t)s * a.max_pages;
      for (int i = 0; i < shared; ++i) stab[i] = ptab[i];
      for (int i = 0; i < need; ++i) {
        const int k = off + i;
        const int slot = top - 1 - k;
        const int pg = slot >= 0 ? a.free_stack[slot] : 0;
        stab[shared + i] = pg;
        a.copy_pairs[2 * k] = ptab[shared + i];
        a.copy_pairs[2 * k + 1] = pg;
      }
    }
    carry += tot;
  }
  __syncthreads();
  if (tid == 0) {
    if (carry > top) { a.state[2] = 1; a.state[0] = 0; a.state[3] = 0; }
    else { a.state[1] = top - carry; a.state[3] = carry; }
  }
}

// ------------------------------------------------------------------ set-up
__global__ __launch_bounds__(1024) void k_setup_scan(SetupArgs a) {
  __shared__ int lds[17];
  const int tid = threadIdx.x;
  int c_tok = 0, c_seq = 0, c_pg = 0;
  for (int base = 0; base < a.P; base += blockDim.x) {
    const int p = base + tid;
    const int L = p < a.P ? a.plen[p] : 0;
    const int g = p < a.P ? a.G[p] : 0;
    const int np = (L + a.page_tok - 1) / a.page_tok;
    int t1, t2, t3;
    const int o1 = block_excl_scan(L, lds, &t1) + c_tok;
    const int o2 = block_excl_scan(g, lds, &t2) + c_seq;
    const int o3 = block_excl_scan(np, lds, &t3) + c_pg;
    if (p < a.P) {
      a.prompt_off[p] = o1;
      a.grp_off[p] = o2;
      a.last_rows[p] = o1 + L - 1;
      int32_t* tab = a.page_tab + (int64_t)(a.n_seq + p) * a.max_pages;
      for (int i = 0; i < np; ++i) tab[i] = o3 + i;   // prompt p's pages are consecutive
    }
    c_tok += t1; c_seq += t2; c_pg += t3;
  }
  if (tid == 0) {
    a.prompt_off[a.P] = c_tok;
    a.grp_off[a.P] = c_seq;
    const bool oom = (int64_t)c_pg > a.pool_pages;
    a.state[0] = oom ? 0 : a.n_seq;
    a.state[1] = oom ? 0 : (int)(a.pool_pages - c_pg);
    a.state[2] = oom ? 1 : 0;
    a.state[3] = 0;
    a.state[4] = c_pg;
    a.state[5] = oom ? 0 : c_tok;   // no prefill rows (so no page writes) without room
    a.state[6] = oom ? 0 : a.P;
    a.state[7] = 0;
    a.state[8] = 0;
  }
}

__global__ void k_setup_free(int32_t* free_stack, const int32_t* state, int64_t pool_pages) {
  const int64_t used = state[4];
  const int64_t n = pool_pages - used;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    free_stack[i] = (int32_t)(used + i);
}

__global__ void k_setup_out(int32_t* tokens, float* logprobs, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    if (tokens) tokens[i] = -1;
    logprobs[i] = 0.f;
  }
}

// ------------------------------------------------------------------ advantage
// One block of 1024 threads.  Pass 1 validates G (every entry >= 1, sum = N).
// Pass 2 walks tiles of 1024 groups: the block scan gives each group its
// offset, then each wave takes groups in turn and reduces them in fp64.
__global__ __launch_bounds__(1024) void k_group_advantage(const float* __restrict__ rewards,
                                                          const int32_t* __restrict__ G, int P, int N, double eps,
                                                          int ddof, float* __restrict__ adv) {
  __shared__ int lds[17];
  __shared__ int offs[1025];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  if (!groups_valid(G, P, N)) {
    for (int i = tid; i < N; i += blockDim.x) adv[i] = __int_as_float(0x7FC00000);
    return;
  }
  int carry = 0;
  for (int base = 0; base < P; base += blockDim.x) {
    const int p = base + tid;
    const int g = p < P ? G[p] : 0;
    int t;
    const int o = block_excl_scan(g, lds, &t) + carry;
    offs[tid] = o;
    if (tid == blockDim.x - 1) offs[blockDim.x] = o + g;
    __syncthreads();
    const int ng = min((int)blockDim.x, P - base);
    for (int k = wave; k < ng; k += nw) {
      const int o0 = offs[k], gs = offs[k + 1] - offs[k];
      const float r0 = rewards[o0];
      double sum = 0.0;
      int diff = 0;
      for (int i = lane; i < gs; i += 64) {
        const float v = rewards[o0 + i];
        sum += (double)v;
        diff |= (v != r0);
      }
      sum = wave_sum_d(sum);
      const bool varies = __any(diff);
      if (!varies || gs - ddof <= 0) {
        for (int i = lane; i < gs; i += 64) adv[o0 + i] = 0.f;
        continue;
      }
      const double mu = sum / (double)gs;
      double sq = 0.0;
      for (int i = lane; i < gs; i += 64) {
        const double dv = (double)rewards[o0 + i] - mu;
        sq += dv * dv;
      }
      sq = wave_sum_d(sq);
      const double sigma = sqrt(sq / (double)(gs - ddof));
      for (int i = lane; i < gs; i += 64) adv[o0 + i] = (float)(((double)rewards[o0 + i] - mu) / (sigma + eps));
    }
    carry += t;
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, int rows_ub, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  if (a.n_slices < 1 || a.V % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_sample_slice, dim3(a.n_slices, rows_ub), dim3(SAMPLE_THREADS), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_sample_pick, dim3(rows_ub), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_compact(const CompactArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_fork(const ForkArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_fork, dim3(1), dim3(1024), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_setup(const SetupArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_setup_scan, dim3(1), dim3(1024), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_setup_free, dim3(1024), dim3(256), 0, st, a.free_stack, a.state, a.pool_pages);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n = (int64_t)a.n_seq * a.max_new;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_setup_out, dim3((unsigned)blocks), dim3(256), 0, st, a.tokens_out, a.logprobs_out, n);
  return hipGetLastError();
}

// ------------------------------------------------------------------ group length statistics
// One 256-thread block per group: the group's offset is the sum of the sizes
// before it; its lengths are ranked in LDS (rank = smaller values plus equal
// values earlier in the group) and placed in sorted order.
__global__ __launch_bounds__(256) void k_group_stats(const int32_t* __restrict__ lengths, const int32_t* __restrict__ G,
                                                     int P, int N, double tau, float* __restrict__ stats) {
  constexpr int GMAX = 1024;
  __shared__ int s_len[GMAX], s_sorted[GMAX];
  __shared__ unsigned long long s_off;
  const int p = blockIdx.x, tid = threadIdx.x;
  if (tid == 0) s_off = 0;
  __syncthreads();
  unsigned long long part = 0;
  for (int i = tid; i < p; i += blockDim.x) part += (unsigned long long)(long long)G[i];
  atomicAdd(&s_off, part);   // integer sum modulo 2^64: order-independent, exact for int32 sizes
  __syncthreads();
  const long long off = (long long)s_off;
  const int g = G[p];
  float* out = stats + 4 * (int64_t)p;
  if (g < 1 || g > GMAX || off < 0 || off + g > N) {
    if (tid < 4) out[tid] = NAN;
    return;
  }
  for (int i = tid; i < g; i += blockDim.x) s_len[i] = lengths[off + i];
  __syncthreads();
  for (int i = tid; i < g; i += blockDim.x) {
    const int v = s_len[i];
    int rank = 0;
    for (int j = 0; j < g; ++j) {
      const int u = s_len[j];
      rank += (u < v) || (u == v && j < i);
    }
    s_sorted[rank] = v;
  }
  __syncthreads();
  if (tid == 0) {
    const int lmax = s_sorted[g - 1];
    const double med = (g & 1) ? (double)s_sorted[g / 2] : ((double)s_sorted[g / 2 - 1] + (double)s_sorted[g / 2]) / 2.0;
    if (!(med > 0.0)) {
      out[0] = out[1] = out[2] = out[3] = NAN;
      return;
    }
    const double R = (double)lmax / med;
    out[0] = (float)lmax;
    out[1] = (float)med;
    out[2] = (float)R;
    out[3] = R > tau ? 1.f : 0.f;
  }
}

hipError_t launch_group_stats(const int32_t* lengths, const int32_t* G, int P, int N, double tau, float* stats,
                              hipStream_t st) {
  if (P < 1) return hipSuccess;
  hipLaunchKernelGGL(k_group_stats, dim3(P), dim3(256), 0, st, lengths, G, P, N, tau, stats);
  return hipGetLastError();
}

// ------------------------------------------------------------------ zero-variance filter
// One block of 1024 threads.  Validates G as the advantage does; then, per
// tile of 1024 groups, the block scan gives each group its offset, one thread
// per group compares its rewards with the first one (exact fp32 equality),
// and a second scan compacts the ids of the groups that vary.  n_kept[0] =
// number of kept groups, or -1 when G is invalid (nothing else written).
__global__ __launch_bounds__(1024) void k_group_filter(const float* __restrict__ rewards, const int32_t* __restrict__ G,
                                                      int P, int N, int32_t* __restrict__ keep,
                                                      int32_t* __restrict__ kept_ids, int32_t* __restrict__ n_kept) {
  __shared__ int lds[17];
  const int tid = threadIdx.x;
  if (!groups_valid(G, P, N)) {
    if (tid == 0) n_kept[0] = -1;
    return;
  }
  int carry = 0, kcarry = 0;
  for (int base = 0; base < P; base += blockDim.x) {
    const int p = base + tid;
    const int g = p < P ? G[p] : 0;
    int t, kt;
    const int o = block_excl_scan(g, lds, &t) + carry;
    int varies = 0;
    if (p < P) {
      const float r0 = rewards[o];
      for (int i = 1; i < g && !varies; ++i) varies = rewards[o + i] != r0;
      keep[p] = varies;
    }
    const int k = block_excl_scan(varies, lds, &kt) + kcarry;
    if (varies) kept_ids[k] = p;
    carry += t;
    kcarry += kt;
  }
  if (tid == 0) n_kept[0] = kcarry;
}

hipError_t launch_group_filter(const float* rewards, const int32_t* G, int P, int N, int32_t* keep, int32_t* kept_ids,
                               int32_t* n_kept, hipStream_t st) {
  hipLaunchKernelGGL(k_group_filter, dim3(1), dim3(1024), 0, st, rewards, G, P, N, keep, kept_ids, n_kept);
  return hipGetLastError();
}

hipError_t launch_group_advantage(const float* rewards, const int32_t* G, int P, int N, float eps, int ddof,
                                  float* adv, hipStream_t st) {
  hipLaunchKernelGGL(k_group_advantage, dim3(1), dim3(1024), 0, st, rewards, G, P, N, (double)eps, ddof, adv);
  return hipGetLastError();
}
