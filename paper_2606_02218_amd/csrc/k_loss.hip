// GRPO loss forward: the row set-up of the teacher-forced log-probability
// recompute over finished rollouts, the per-token log-probability gather
// after the lm head, and the clipped surrogate reduction.
#include <mutex>
#include <vector>

#include "rg_device.h"
#include "rg_kernels.h"

// Scratch of grpo_surrogate_noalloc: the per-sequence records of up to
// SURROGATE_NOALLOC_MAX_SEQS sequences (1 MiB), one copy on every device the
// library runs on, held until the process ends.  Host code never passes this
// name to a kernel: it uses the device address surrogate_static_scratch()
// looks up.
static __device__ __align__(256) SurrogateRec scratch[SURROGATE_NOALLOC_MAX_SEQS];

namespace {

// One block of 1024 threads, after the fork.  Per sequence s (lengths checked
// to lie in [1, max_new]): coff[s] = exclusive prefix of L_s - 1, the start of
// its rows among all teacher-forced rows; and fresh pages, popped from the
// free stack, for the positions plen + 0 .. plen + L_s - 2 that the forward
// writes.  coff[n_seq] and state[9] get the row total, state[10] = 1 if a
// length was out of range, state[2] = 1 if the pool ran out (page tables are
// then not usable).
__global__ __launch_bounds__(1024) void k_reserve(ReserveArgs a) {
  __shared__ int lds[17];
  __shared__ int s_bad;
  const int tid = threadIdx.x;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  const int top = a.state[1];
  int rcarry = 0, pcarry = 0;
  for (int base = 0; base < a.n_seq; base += blockDim.x) {
    const int s = base + tid;
    int rows = 0, need = 0, have = 0;
    if (s < a.n_seq) {
      int L = a.lengths[s];
      if (L < 1 || L > a.max_new) {
        atomicOr(&s_bad, 1);
        L = 1;
      }
      const int ctx = a.plen[a.seq_grp[s]] + L - 1;   // positions holding keys and values
      have = a.seq_npages[s];
      need = max(0, (ctx + a.page_tok - 1) / a.page_tok - have);
      rows = L - 1;
    }
    int rt, pt;
    const int ro = block_excl_scan(rows, lds, &rt) + rcarry;
    const int po = block_excl_scan(need, lds, &pt) + pcarry;
    if (s < a.n_seq) {
      a.coff[s] = ro;
      int32_t* tab = a.page_tab + (int64_t)s * a.max_pages;
      for (int i = 0; i < need; ++i) {
        const int slot = top - 1 - (po + i);
        tab[have + i] = slot >= 0 ? a.free_stack[slot] : 0;
      }
      a.seq_npages[s] = have + need;
    }
    rcarry += rt;
    pcarry += pt;
  }
  if (tid == 0) {
    a.coff[a.n_seq] = rcarry;
    a.state[9] = rcarry;
    a.state[10] = s_bad;
    if (pcarry > top) a.state[2] = 1;
    else a.state[1] = top - pcarry;
  }
}

// Rows row0 .. row0 + gridDim.x - 1 of the teacher-forced forward.  Global row
// g belongs to the sequence s with coff[s] <= g < coff[s + 1] and feeds token
// y_t, t = g - coff[s], at position plen + t; it predicts y_{t+1}, whose
// log-probability lands in logprobs[s * max_new + t + 1].
template <typename T>
__global__ __launch_bounds__(256) void k_recompute_rows(RecomputeRows a, const T* __restrict__ embed) {
  const int r = blockIdx.x;
  const int g = a.row0 + r;
  int lo = 0, hi = a.n_seq - 1;   // last s with coff[s] <= g: never an empty sequence
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.coff[mid] <= g) lo = mid; else hi = mid - 1;
  }
  const int s = lo;
  const int t = g - a.coff[s];
  const int64_t o = (int64_t)s * a.max_new + t;
  int tok = a.tokens[o];
  if (tok < 0 || tok >= a.V) {
    if (threadIdx.x == 0) a.bad_token[0] = 1;
    tok = 0;
  }
  if (threadIdx.x == 0) {
    int tgt = a.tokens[o + 1];
    if (tgt < 0 || tgt >= a.V) {
      a.bad_token[0] = 1;
      tgt = 0;
    }
    a.row_tab[r] = s;
    a.row_pos[r] = a.plen[a.seq_grp[s]] + t;
    a.row_beg[r] = 0;
    a.row_tgt[r] = tgt;
    a.row_out[r] = (int32_t)(o + 1);
  }
  const T* e = embed + (int64_t)tok * a.d;
  for (int i = threadIdx.x; i < a.d; i += blockDim.x) a.x[(int64_t)r * a.d + i] = ld_f32<T>(e + i);
}

// Tiles of the chunk's rows for the row-tile attention: each sequence's rows
// in the chunk, cut into runs of tr from its first row.  One block of 1024
// threads; tile k starts at row tile_r0[k] and has tile_nr[k] rows, in row
// order; *d_tiles gets the count.
__global__ __launch_bounds__(1024) void k_row_tiles(const int32_t* __restrict__ row_tab,
                                                    const int32_t* __restrict__ coff, int row0, int n, int tr,
                                                    int32_t* __restrict__ tile_r0, int32_t* __restrict__ tile_nr,
                                                    int* __restrict__ d_tiles) {
  __shared__ int lds[17];
  int carry = 0;
  for (int base = 0; base < n; base += blockDim.x) {
    const int r = base + threadIdx.x;
    int flag = 0, len = 0;
    if (r < n) {
      const int s = row_tab[r];
      const int f = max(coff[s] - row0, 0);         // the sequence's first row in this chunk
      const int e = min(coff[s + 1] - row0, n);     // one past its last
      flag = (r - f) % tr == 0;
      len = min(tr, e - r);
    }
    int tot;
    const int o = block_excl_scan(flag, lds, &tot) + carry;
    if (flag) {
      tile_r0[o] = r;
      tile_nr[o] = len;
    }
    carry += tot;
  }
  if (threadIdx.x == 0) *d_tiles = carry;
}

// Step 0 of every sequence: its prompt's last-position logits (row seq_grp[s])
// score y_0, stored at logprobs[s * max_new].
__global__ void k_first_rows(const int32_t* __restrict__ tokens, const int32_t* __restrict__ seq_grp, int n_seq,
                             int max_new, int V, int32_t* __restrict__ lrow, int32_t* __restrict__ tgt,
                             int32_t* __restrict__ out, int32_t* __restrict__ bad_token) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_seq) return;
  int y = tokens[(int64_t)s * max_new];
  if (y < 0 || y >= V) {
    bad_token[0] = 1;
    y = 0;
  }
  lrow[s] = seq_grp[s];
  tgt[s] = y;
  out[s] = s * max_new;
}

// One block per row: logsumexp of z/T over the full vocabulary (the running
// (max, sum) form the sampler uses, in fp32), then
// lp[out[r]] = z[tgt[r]]/T - logsumexp.  z = logits row lrow[r] (or r).
constexpr int LP_THREADS = 256;

__global__ __launch_bounds__(LP_THREADS) void k_token_logprob(const float* __restrict__ logits, int V, float T,
                                                            const int32_t* __restrict__ lrow,
                                                            const int32_t* __restrict__ tgt,
                                                            const int32_t* __restrict__ out, float* __restrict__ lp) {
  const int r = blockIdx.x, tid = threadIdx.x;
  const float* z = logits + (int64_t)(lrow ? lrow[r] : r) * V;
  float m = -INFINITY, sum = 0.f;
  for (int v = tid * 4; v < V; v += LP_THREADS * 4) {
    const float4 zz = *reinterpret_cast<const float4*>(z + v);
    const float e[4] = {zz.x, zz.y, zz.z, zz.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float zt = e[j] / T;
      if (zt > m) { sum = sum * expf(m - zt) + 1.f; m = zt; }
      else sum += expf(zt - m);
    }
  }
  __shared__ float sm[LP_THREADS], ss[LP_THREADS];
  sm[tid] = m;
  ss[tid] = sum;
  __syncthreads();
  for (int o = LP_THREADS / 2; o > 0; o >>= 1) {
    if (tid < o) {
      const float m1 = sm[tid], m2 = sm[tid + o];
      const float mm = fmaxf(m1, m2);
      ss[tid] = (m1 == -INFINITY ? 0.f : ss[tid] * expf(m1 - mm)) + (m2 == -INFINITY ? 0.f : ss[tid + o] * expf(m2 - mm));
      sm[tid] = mm;
    }
    __syncthreads();
  }
  if (tid == 0) lp[out[r]] = z[tgt[r]] / T - (sm[0] + logf(ss[0]));
}

// Clipped surrogate, pass 1: one wave per sequence s < N.  Its lanes stride
// over the sequence's L_s tokens and accumulate, in fp64,
// min(rho * A_s, clip(rho, 1 - eps_lo, 1 + eps_hi) * A_s), rho = exp(new - old),
// then the wave sums them (a butterfly: a fixed order).  rec[s] = (sum,
// clipped tokens); a length outside [1, max_new] writes clipped = -1.
__global__ __launch_bounds__(256) void k_surrogate_seq(SurrogateArgs a, SurrogateRec* __restrict__ rec) {
  const int lane = threadIdx.x & 63;
  const int s = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (s >= a.N) return;
  const int L = a.lengths[s];
  if (L < 1 || L > a.max_new) {
    if (lane == 0) rec[s] = SurrogateRec{0.0, -1, 0};
    return;
  }
  const double A = (double)a.adv[s];
  const int64_t row = (int64_t)s * a.max_new;
  double acc = 0.0;
  int clips = 0;
  for (int i = lane; i < L; i += 64) {
    const double rho = exp((double)a.new_lp[row + i] - (double)a.old_lp[row + i]);
    const double un = rho * A;
    const double cl = fmin(fmax(rho, 1.0 - a.eps_lo), 1.0 + a.eps_hi) * A;
    acc += fmin(un, cl);
    clips += cl < un;
  }
  acc = wave_sum_d(acc);
  for (int o = 32; o > 0; o >>= 1) clips += __shfl_xor(clips, o, 64);
  if (lane == 0) rec[s] = SurrogateRec{acc, clips, 0};
}

// Pass 2, one block of 1024 threads: the group partition (each G[p] >= 1,
// sum N), then thread t takes groups t, t + 1024, ... whose keep flag is set
// and adds their members' records in sequence order; the per-thread totals
// are combined by a butterfly within each wave and the wave totals in wave
// order, so the result does not depend on timing.  out = (loss, clipped
// fraction, tokens, sequences); NaN in all four for an invalid partition or
// a length outside [1, max_new], zeros when nothing is counted.
__global__ __launch_bounds__(1024) void k_surrogate_reduce(SurrogateArgs a, const SurrogateRec* __restrict__ rec) {
  __shared__ int lds[17];
  __shared__ double w_tok[16], w_seq[16];
  __shared__ long long w_ntok[16], w_nclip[16];
  __shared__ int w_nseq[16], w_bad[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  if (!groups_valid(a.G, a.P, a.N)) {
    if (tid < 4) a.out[tid] = __longlong_as_double(0x7FF8000000000000ll);
    return;
  }
  double tok_sum = 0.0, seq_sum = 0.0;
  long long n_tok = 0, n_clip = 0;
  int n_seq = 0, bad = 0;
  int carry = 0;
  for (int base = 0; base < a.P; base += blockDim.x) {
    const int p = base + tid;
    const int g = p < a.P ? a.G[p] : 0;
    int t;
    const int o = block_excl_scan(g, lds, &t) + carry;
    if (p < a.P && (!a.keep || a.keep[p] != 0)) {
      for (int s = o; s < o + g; ++s) {
        const SurrogateRec r = rec[s];
        if (r.clips < 0) {
          bad = 1;
          continue;
        }
        const int L = a.lengths[s];
        tok_sum += r.acc;
        seq_sum += r.acc / (double)L;
        n_tok += L;
        n_clip += r.clips;
        n_seq += 1;
      }
    }
    carry += t;
  }
  tok_sum = wave_sum_d(tok_sum);
  seq_sum = wave_sum_d(seq_sum);
  for (int o = 32; o > 0; o >>= 1) {
    n_tok += __shfl_xor(n_tok, o, 64);
    n_clip += __shfl_xor(n_clip, o, 64);
    n_seq += __shfl_xor(n_seq, o, 64);
    bad |= __shfl_xor(bad, o, 64);
  }
  if (lane == 0) {
    w_tok[wave] = tok_sum; w_seq[wave] = seq_sum; w_ntok[wave] = n_tok; w_nclip[wave] = n_clip;
    w_nseq[wave] = n_seq; w_bad[wave] = bad;
  }
  __syncthreads();
  if (tid == 0) {
    double ts = 0.0, qs = 0.0;
    long long nt = 0, nc = 0;
    int ns = 0, nb = 0;
    for (int w = 0; w < nw; ++w) {
      ts += w_tok[w]; qs += w_seq[w]; nt += w_ntok[w]; nc += w_nclip[w]; ns += w_nseq[w]; nb |= w_bad[w];
    }
    if (nb) {
      for (int i = 0; i < 4; ++i) a.out[i] = __longlong_as_double(0x7FF8000000000000ll);
    } else if (ns == 0) {
      for (int i = 0; i < 4; ++i) a.out[i] = 0.0;
    } else {
      const double agg = a.mode == 0 ? ts / (double)nt : qs / (double)ns;
      a.out[0] = -agg;
      a.out[1] = (double)nc / (double)nt;
      a.out[2] = (double)nt;
      a.out[3] = (double)ns;
    }
  }
}

}  // namespace

hipError_t launch_reserve(const ReserveArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_reserve, dim3(1), dim3(1024), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_recompute_rows(int dtype, const void* embed, const RecomputeRows& a, int rows, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(k_recompute_rows<bf16_t>, dim3(rows), dim3(256), 0, st, a, (const bf16_t*)embed);
  else
    hipLaunchKernelGGL(k_recompute_rows<float>, dim3(rows), dim3(256), 0, st, a, (const float*)embed);
  return hipGetLastError();
}

hipError_t launch_row_tiles(const int32_t* row_tab, const int32_t* coff, int row0, int n, int tile_rows,
                            int32_t* tile_r0, int32_t* tile_nr, int* d_tiles, hipStream_t st) {
  hipLaunchKernelGGL(k_row_tiles, dim3(1), dim3(1024), 0, st, row_tab, coff, row0, n, tile_rows, tile_r0, tile_nr,
                     d_tiles);
  return hipGetLastError();
}

hipError_t launch_first_rows(const int32_t* tokens, const int32_t* seq_grp, int n_seq, int max_new, int V,
                             int32_t* lrow, int32_t* tgt, int32_t* out, int32_t* bad_token, hipStream_t st) {
  hipLaunchKernelGGL(k_first_rows, dim3((n_seq + 255) / 256), dim3(256), 0, st, tokens, seq_grp, n_seq, max_new, V,
                     lrow, tgt, out, bad_token);
  return hipGetLastError();
}

hipError_t launch_token_logprob(const float* logits, int V, float T, const int32_t* lrow, const int32_t* tgt,
                                const int32_t* out, float* lp, int rows, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_token_logprob, dim3(rows), dim3(LP_THREADS), 0, st, logits, V, T, lrow, tgt, out, lp);
  return hipGetLastError();
}

hipError_t surrogate_static_scratch(SurrogateRec** out) {
  static std::mutex mu;
  static std::vector<SurrogateRec*> by_device;   // device address of `scratch`, per device
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)by_device.size() <= dev) by_device.resize(dev + 1, nullptr);
  if (!by_device[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    by_device[dev] = (SurrogateRec*)ptr;
  }
  *out = by_device[dev];
  return hipSuccess;
}

hipError_t launch_surrogate(const SurrogateArgs& a, SurrogateRec* rec, hipStream_t st) {
  if (a.N < 1 || !rec) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_surrogate_seq, dim3((a.N + 3) / 4), dim3(256), 0, st, a, rec);
  hipLaunchKernelGGL(k_surrogate_reduce, dim3(1), dim3(1024), 0, st, a, (const SurrogateRec*)rec);
  return hipGetLastError();
}
